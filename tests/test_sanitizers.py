"""AddressSanitizer / UBSan runs of host code (CPU only, test infrastructure).

- The C ABI's host paths: fma_api.hip is built with the host side
  instrumented (-Xarch_host before each sanitizer flag; its device side
  holds only the static scratch buffer) and linked with launcher stubs that
  abort if reached; tests/sanitize/host_api_check.c then builds plans across
  the supported space, queries every size and the plan-parameter export, and
  drives every validation path of every entry point (no launch is reached).
- The C oracle: built serially with gcc's sanitizers and driven by
  tests/sanitize/oracle_check.c on small 1D / 2D problems with exactly sized
  buffers, checking weights-sum-to-one, causality and the backward.
Either run fails on any sanitizer report.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
INC = os.path.join(ROOT, "include")
CSRC = os.path.join(ROOT, "paper_2310_11960_amd", "csrc")
HIPCC = "/opt/rocm/bin/hipcc"
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), r.stdout[-3000:], r.stderr[-3000:])
    return r


@pytest.mark.skipif(not os.path.exists(HIPCC) or shutil.which("gcc") is None, reason="needs hipcc and gcc")
def test_host_api_under_sanitizers(tmp_path):
    d = str(tmp_path)
    common = ["-O1", "-g", "-std=c++17", "--offload-arch=gfx950", "-fno-omit-frame-pointer", "-I", INC, "-I", CSRC]
    _run([HIPCC, *common, *HOST_SAN, "-c", os.path.join(CSRC, "fma_api.hip"), "-o", d + "/api.o"])
    _run([HIPCC, *common, "--cuda-host-only", *HOST_SAN, "-c", os.path.join(SAN, "launch_stubs.hip"),
          "-o", d + "/stubs.o"])
    _run(["gcc", "-O1", "-g", "-std=c11", "-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-I", INC,
          "-c", os.path.join(SAN, "host_api_check.c"), "-o", d + "/driver.o"])
    _run([HIPCC, "--offload-arch=gfx950", *HOST_SAN, d + "/driver.o", d + "/api.o", d + "/stubs.o",
          "-o", d + "/host_check"])
    r = _run([d + "/host_check"], env=ENV)
    assert "host api checks passed" in r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_check")
    _run(["gcc", "-O1", "-g", "-std=c11", "-Wall", "-Wno-unknown-pragmas", "-fsanitize=address,undefined",
          "-fno-omit-frame-pointer", os.path.join(ROOT, "oracle", "fma_oracle.c"),
          os.path.join(SAN, "oracle_check.c"), "-lm", "-o", exe])
    r = _run([exe], env=ENV)
    assert "oracle checks passed" in r.stdout
