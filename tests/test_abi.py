"""Host-side tests of the C ABI: the library loads, exports everything the
header declares, and validates arguments before touching the device.

No call here reaches a kernel launch: every call that is given (fake)
device pointers is built to fail validation first.
"""
import ctypes
import os
import subprocess
import tempfile

import pytest
import torch

import oracle
import paper_2310_11960_amd as F


def test_library_exports_every_header_function():
    lib = F.library()
    names = F.header_functions()
    assert "fma_plan" in names and "fma_forward_1d" in names and "fma_forward_2d" in names
    for n in names:
        assert hasattr(lib, n), n


def test_desc_layout_matches_header():
    """The binding's struct has the size and field offsets the C compiler
    gives the header's fma_desc_t."""
    names = [f[0] for f in F.fma_desc_t._fields_]
    src = '#include <stdio.h>\n#include <stddef.h>\n#include "fma.h"\nint main(void){\n'
    src += 'printf("size %zu\\n", sizeof(fma_desc_t));\n'
    for n in names:
        src += 'printf("%s %%zu\\n", offsetof(fma_desc_t, %s));\n' % (n, n)
    src += "return 0;}\n"
    with tempfile.TemporaryDirectory() as td:
        c, exe = os.path.join(td, "probe.c"), os.path.join(td, "probe")
        open(c, "w").write(src)
        subprocess.run(["gcc", "-I", os.path.dirname(F.HEADER_PATH), c, "-o", exe], check=True)
        out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout.split()
    got = dict(zip(out[0::2], map(int, out[1::2])))
    assert got["size"] == ctypes.sizeof(F.fma_desc_t)
    for n in names:
        assert got[n] == getattr(F.fma_desc_t, n).offset, n


@pytest.mark.parametrize("n,r", [(1024, 64), (4096, 64), (16384, 128), (65536, 128), (768, 64),
                                 (1280, 128), (64, 64), (128, 64), (3 * 256, 256), (192 * 5, 192)])
def test_geometry_1d(n, r):
    op = F.FMA(ndim=1, batch=2, heads=3, seq_len=n, block=r)
    assert op.levels == oracle.num_levels(n // r)
    assert op.coarse_rows == oracle.coarse_rows_1d(n, r)
    L = op.levels
    assert op.weights_len == sum(r * 2 ** (l - 1) for l in range(1, L))
    if L > 1:
        R = op.coarse_rows
        assert op.workspace_bytes >= 2 * 2 * 3 * R * 64 * 2
    else:
        assert op.workspace_bytes == 0


@pytest.mark.parametrize("W,r", [(128, 8), (64, 16), (24, 8), (40, 8), (16, 8), (8, 8), (256, 16)])
def test_geometry_2d(W, r):
    op = F.FMA(ndim=2, batch=1, heads=2, seq_len=W * W, block=r, side=W)
    assert op.levels == oracle.num_levels(W // r)
    assert op.coarse_rows == oracle.coarse_rows_2d(W, r)
    assert op.weights_len == sum(2 * r * 2 ** (l - 1) for l in range(1, op.levels))


@pytest.mark.parametrize("H,W,r,p", [(32, 64, 8, 1), (128, 32, 8, 1), (24, 40, 8, 2), (8, 64, 8, 1), (48, 16, 4, 1),
                                     (64, 128, 16, 3)])
def test_geometry_2d_rect(H, W, r, p):
    """Maps of H rows by W columns: the depth follows the longer side, and
    the plan's cell and square counts follow each axis."""
    op = F.FMA(ndim=2, batch=1, heads=2, seq_len=H * W, block=r, side=W, rank=p)
    assert op.levels == oracle.num_levels(max(H, W) // r) == oracle.levels_2d(W, r, H=H)
    assert op.coarse_rows == p * oracle.coarse_rows_2d(W, r, H=H)
    assert op.weights_len == oracle.weight_len_2d(W, r, p, H=H)
    P = F.fma_plan_params(op.handle)
    assert (P["height"], P["nbx"], P["nby"], P["tiles_per_slice"]) == (H, H // r, W // r, (H // r) * (W // r))
    for st in P["sets"]:
        s = st["size"]
        assert (st["M"], st["My"]) == (-(-H // s), -(-W // s))


def test_backward_workspace_bounded():
    """The backward's per-workgroup coarse partials are kept for a pass of
    slices at a time (192 MiB), so the workspace does not grow with a
    partial row per slice of the whole batch: every workload's backward
    needs under 0.5 GiB (C5 needed 1.46 GB with partials for all slices)."""
    import fma_inputs
    for name in ("C2", "C3", "C4", "C5"):
        w = fma_inputs.WORKLOADS[name]
        op = F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block, causal=w.causal,
                   dtype=w.torch_dtype, side=w.side)
        assert op.backward_workspace_bytes < 512 << 20, (name, op.backward_workspace_bytes)


def _status(fn):
    with pytest.raises(F.FmaError) as e:
        fn()
    return e.value.status


def test_plan_rejections():
    mk = lambda **kw: F.FMA(**{**dict(ndim=1, batch=1, heads=1, seq_len=1024, block=64), **kw})
    assert _status(lambda: mk(seq_len=1000)) == F.FMA_ERR_SHAPE            # r does not divide n
    assert _status(lambda: mk(head_dim=96)) == F.FMA_ERR_UNSUPPORTED     # 32, 64 and 128 are built
    assert _status(lambda: mk(head_dim=16)) == F.FMA_ERR_UNSUPPORTED
    for d in (32, 128):
        op = mk(head_dim=d)
        assert F.fma_plan_params(op.handle)["head_dim"] == d
        # the backward is built for d = 64 only
        assert _status(lambda: F.fma_backward(op.handle, *[FAKE * (i + 1) for i in range(12)], FAKE * 256,
                                              op.backward_workspace_bytes, 0)) == F.FMA_ERR_UNSUPPORTED
    assert _status(lambda: mk(block=48, seq_len=48 * 16)) == F.FMA_ERR_UNSUPPORTED
    assert _status(lambda: mk(block=8)) == F.FMA_ERR_UNSUPPORTED
    assert _status(lambda: mk(block=512, seq_len=4096)) == F.FMA_ERR_UNSUPPORTED
    assert _status(lambda: mk(num_levels=3)) == F.FMA_ERR_SHAPE            # L is 4
    assert _status(lambda: mk(ndim=3)) == F.FMA_ERR_ARG
    assert _status(lambda: mk(dtype=7)) == F.FMA_ERR_ARG
    assert _status(lambda: mk(batch=-1)) == F.FMA_ERR_SHAPE
    assert _status(lambda: mk(softmax_scale=float("nan"))) == F.FMA_ERR_ARG
    assert _status(lambda: mk(ndim=2, seq_len=128 * 128, side=128, block=8, causal=True)) == F.FMA_ERR_UNSUPPORTED
    assert _status(lambda: mk(ndim=2, seq_len=100, side=12, block=8)) == F.FMA_ERR_SHAPE
    assert _status(lambda: mk(ndim=2, seq_len=144, side=12, block=8)) == F.FMA_ERR_SHAPE
    assert _status(lambda: mk(ndim=2, seq_len=12 * 40, side=40, block=8)) == F.FMA_ERR_SHAPE   # r does not divide H
    assert _status(lambda: mk(ndim=2, seq_len=64 * 60, side=60, block=8)) == F.FMA_ERR_SHAPE   # r does not divide W
    assert _status(lambda: mk(ndim=2, seq_len=256, side=-1, block=8)) == F.FMA_ERR_SHAPE
    assert _status(lambda: mk(ndim=2, seq_len=16 * 16, side=16, block=2)) == F.FMA_ERR_UNSUPPORTED
    # blocks of 16 and 32 tokens (1D) and 4 x 4 cells (2D) plan; their backward is not built
    assert mk(block=16).levels == 6 and mk(block=32).levels == 5
    assert mk(ndim=2, seq_len=16 * 16, side=16, block=4).levels == 2
    small = mk(block=16)
    assert _status(lambda: F.fma_backward(small.handle, *[FAKE * (i + 1) for i in range(12)], FAKE * 256,
                                          small.backward_workspace_bytes - 1, 0)) == F.FMA_ERR_WORKSPACE
    # sequence long enough for more coarse levels than the kernels carry
    assert _status(lambda: mk(seq_len=64 << 18)) == F.FMA_ERR_UNSUPPORTED
    assert mk(num_levels=4).levels == 4
    assert "does not divide" in (lambda: (_status(lambda: mk(seq_len=1000)), F.fma_last_error()))()[1]


def test_struct_size_checked():
    d = F.make_desc(seq_len=1024)
    d.struct_size = 12
    assert _status(lambda: F.fma_plan(d)) == F.FMA_ERR_ARG
    # a descriptor that ends before `rank` is a rank-1 plan, whatever follows it
    d = F.make_desc(seq_len=1024, rank=3)
    d.struct_size = F.fma_desc_t.rank.offset
    h = F.fma_plan(d)
    try:
        assert F.fma_weights_len(h) == oracle.weight_len_1d(1024, 64, 1)
    finally:
        F.fma_destroy(h)


@pytest.mark.parametrize("n,r,p", [(1024, 64, 2), (4096, 64, 4), (16384, 128, 4), (65536, 128, 4),
                                   (65536, 128, 8), (768, 64, 3), (64, 64, 5)])
def test_geometry_rank_1d(n, r, p):
    op = F.FMA(ndim=1, batch=2, heads=3, seq_len=n, block=r, rank=p)
    assert op.weights_len == oracle.weight_len_1d(n, r, p)
    assert op.coarse_rows == p * oracle.coarse_rows_1d(n, r)
    if op.levels > 1:
        assert op.workspace_bytes >= 2 * 2 * 3 * op.coarse_rows * 64 * 2


@pytest.mark.parametrize("W,r,p", [(128, 8, 4), (128, 8, 5), (64, 16, 2), (24, 8, 3)])
def test_geometry_rank_2d(W, r, p):
    op = F.FMA(ndim=2, batch=1, heads=2, seq_len=W * W, block=r, side=W, rank=p)
    assert op.weights_len == oracle.weight_len_2d(W, r, p)
    assert op.coarse_rows == p * oracle.coarse_rows_2d(W, r)


def test_norm_validation():
    mk = lambda **kw: F.FMA(**{**dict(ndim=1, batch=1, heads=1, seq_len=4096, block=64), **kw})
    assert _status(lambda: mk(norm=2)) == F.FMA_ERR_ARG
    assert mk(norm=F.FMA_NORM_PER_LEVEL).weights_len == oracle.weight_len_1d(4096, 64, 1)
    assert mk(norm=F.FMA_NORM_PER_LEVEL, rank=10, seq_len=2048).coarse_rows == 10 * oracle.coarse_rows_1d(2048, 64)
    # 3 * 11 = 33 slots per level do not fit one 32-key group
    assert _status(lambda: mk(norm=F.FMA_NORM_PER_LEVEL, rank=11, seq_len=1024)) == F.FMA_ERR_UNSUPPORTED
    # 2D per-level: 27 slots pad to 32; rank p >= 2 pads 27p to a multiple of 32
    # (whole blocks per level), and levels x slots must fit the 448-slot table
    for p_, grp in ((1, 32), (2, 64), (3, 96), (4, 128), (5, 160)):
        op = mk(ndim=2, seq_len=64 * 64, side=64, block=8, norm=F.FMA_NORM_PER_LEVEL, rank=p_)
        P = F.fma_plan_params(op.handle)
        assert (P["slot_group"], P["nslot"]) == (grp, grp * (op.levels - 1)), p_
    assert _status(lambda: mk(ndim=2, seq_len=128 * 128, side=128, block=8, norm=F.FMA_NORM_PER_LEVEL,
                              rank=5)) == F.FMA_ERR_UNSUPPORTED   # 3 levels x 160 slots
    # 2D joint: 4 levels x 5 bases x 27 squares = 540 slots exceed the 448-slot table
    assert _status(lambda: mk(ndim=2, seq_len=256 * 256, side=256, block=8, rank=5)) == F.FMA_ERR_UNSUPPORTED
    assert mk(ndim=2, seq_len=256 * 256, side=256, block=8, rank=4).coarse_rows == 4 * oracle.coarse_rows_2d(256, 8)


def test_linear_plans():
    mk = lambda **kw: F.FMA(**{**dict(ndim=1, batch=1, heads=1, seq_len=4096, block=64), **kw})
    assert _status(lambda: mk(linear=True, causal=True)) == F.FMA_ERR_UNSUPPORTED
    assert _status(lambda: mk(linear=True, rank=2)) == F.FMA_ERR_UNSUPPORTED
    assert _status(lambda: mk(linear=True, norm=F.FMA_NORM_PER_LEVEL)) == F.FMA_ERR_UNSUPPORTED
    lin, std = mk(linear=True), mk()
    assert lin.workspace_bytes > std.workspace_bytes
    ws = lin.workspace_bytes
    # the plain forward rejects a linear plan and the linear forward a plain one
    assert _status(lambda: F.fma_forward_1d(lin.handle, FAKE, FAKE * 2, FAKE * 3, FAKE * 4, FAKE * 5, FAKE * 8,
                                            FAKE * 16, ws, 0)) == F.FMA_ERR_ARG
    assert _status(lambda: F.fma_forward_linear(std.handle, FAKE, FAKE * 2, FAKE * 3, FAKE * 6, FAKE * 4,
                                                FAKE * 5, FAKE * 8, FAKE * 16, ws, 0)) == F.FMA_ERR_ARG
    assert _status(lambda: F.fma_forward_linear(lin.handle, FAKE, FAKE * 2, FAKE * 3, None, FAKE * 4,
                                                FAKE * 5, FAKE * 8, FAKE * 16, ws, 0)) == F.FMA_ERR_NULL
    # FMA-linear plans take fma_backward_linear, and only they do
    assert _status(lambda: F.fma_backward(lin.handle, *[FAKE * (i + 1) for i in range(12)], FAKE * 256,
                                          lin.backward_workspace_bytes, 0)) == F.FMA_ERR_ARG
    assert _status(lambda: F.fma_backward_linear(std.handle, *[FAKE * (i + 1) for i in range(14)], FAKE * 256,
                                                 std.backward_workspace_bytes, 0)) == F.FMA_ERR_ARG
    lb = lin.backward_workspace_bytes
    assert lb > std.backward_workspace_bytes
    assert _status(lambda: F.fma_backward_linear(lin.handle, *[FAKE * (i + 1) for i in range(14)], FAKE * 256,
                                                 lb - 1, 0)) == F.FMA_ERR_WORKSPACE
    args = [FAKE * (i + 1) for i in range(14)]
    args[5] = None                                      # wq
    assert _status(lambda: F.fma_backward_linear(lin.handle, *args, FAKE * 256, lb, 0)) == F.FMA_ERR_NULL
    args = [FAKE * (i + 1) for i in range(14)]
    args[13] = args[0]                                  # dwq aliasing q
    assert _status(lambda: F.fma_backward_linear(lin.handle, *args, FAKE * 256, lb, 0)) == F.FMA_ERR_ARG


def test_rank_rejections():
    mk = lambda **kw: F.FMA(**{**dict(ndim=1, batch=1, heads=1, seq_len=1024, block=64), **kw})
    assert _status(lambda: mk(rank=-1)) == F.FMA_ERR_ARG
    assert mk(rank=0).weights_len == oracle.weight_len_1d(1024, 64, 1)
    # 8 coarse levels x rank 9 = 72 sets > 64
    assert _status(lambda: mk(seq_len=64 << 9, rank=9)) == F.FMA_ERR_UNSUPPORTED
    assert mk(seq_len=64 << 9, rank=8).coarse_rows == 8 * oracle.coarse_rows_1d(64 << 9, 64)
    # 2D: 3 coarse levels x rank 6 = 18 sets > 16
    assert _status(lambda: mk(ndim=2, seq_len=128 * 128, side=128, block=8, rank=6)) == F.FMA_ERR_UNSUPPORTED


FAKE = 0x100000   # 16-byte aligned, never dereferenced: every call below fails validation


def test_forward_validation_before_launch():
    op = F.FMA(ndim=1, batch=1, heads=1, seq_len=4096, block=64)
    h, ws = op.handle, op.workspace_bytes
    f = F.fma_forward_1d
    # NULL tensors
    assert _status(lambda: f(h, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ws, 0)) == F.FMA_ERR_NULL
    # misaligned q
    assert _status(lambda: f(h, FAKE + 2, FAKE, FAKE, FAKE, FAKE, FAKE * 2, FAKE * 3, ws, 0)) == F.FMA_ERR_ALIGN
    # missing weights with coarse levels
    assert _status(lambda: f(h, FAKE, FAKE, FAKE, None, FAKE, FAKE * 8, FAKE * 16, ws, 0)) == F.FMA_ERR_NULL
    # workspace too small / missing
    assert _status(lambda: f(h, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE * 8, FAKE * 16, ws - 1, 0)) == F.FMA_ERR_WORKSPACE
    assert _status(lambda: f(h, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE * 8, None, ws, 0)) == F.FMA_ERR_WORKSPACE
    # out aliasing q
    assert _status(lambda: f(h, FAKE, FAKE * 64, FAKE * 128, FAKE, FAKE, FAKE, FAKE * 256, ws, 0)) == F.FMA_ERR_ARG
    # wrong entry point for the plan's dimensionality
    assert _status(lambda: F.fma_forward_2d(h, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE * 8, FAKE * 16, ws, 0)) == F.FMA_ERR_SHAPE
    # NULL plan
    assert _status(lambda: f(None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ws, 0)) == F.FMA_ERR_NULL
    assert _status(lambda: F.fma_coarsen(h, FAKE, FAKE, None, None, FAKE * 16, ws, 0)) == F.FMA_ERR_NULL
    assert _status(lambda: F.fma_attend(h, FAKE, FAKE, FAKE, None, 0, FAKE * 8, 0)) == F.FMA_ERR_WORKSPACE
    assert _status(lambda: F.fma_interaction_lists(h, None, 0)) == F.FMA_ERR_NULL
    assert _status(lambda: F.fma_dense_reference(h, FAKE, FAKE, FAKE, FAKE, 0)) == F.FMA_ERR_ARG


def test_backward_validation_before_launch():
    op = F.FMA(ndim=1, batch=1, heads=1, seq_len=4096, block=64)
    h, ws = op.handle, op.backward_workspace_bytes
    assert ws > op.workspace_bytes
    f = F.fma_backward
    A = [FAKE * (i + 1) for i in range(8)]     # q, k, v, out, dout, dq, dk, dv: disjoint fakes
    W = [FAKE * 64, FAKE * 65, FAKE * 66, FAKE * 67]   # wk, wv, dwk, dwv
    WS = FAKE * 256
    # NULL plan, NULL tensor, misaligned tensor
    assert _status(lambda: f(None, *A[:3], W[0], W[1], A[3], A[4], *A[5:], W[2], W[3], WS, ws, 0)) == F.FMA_ERR_NULL
    assert _status(lambda: f(h, None, *A[1:3], W[0], W[1], A[3], A[4], *A[5:], W[2], W[3], WS, ws, 0)) == F.FMA_ERR_NULL
    assert _status(lambda: f(h, A[0] + 2, *A[1:3], W[0], W[1], A[3], A[4], *A[5:], W[2], W[3], WS, ws, 0)) == F.FMA_ERR_ALIGN
    # missing weight gradients, small workspace
    assert _status(lambda: f(h, *A[:3], W[0], W[1], A[3], A[4], *A[5:], None, W[3], WS, ws, 0)) == F.FMA_ERR_NULL
    assert _status(lambda: f(h, *A[:3], W[0], W[1], A[3], A[4], *A[5:], W[2], W[3], WS, ws - 1, 0)) == F.FMA_ERR_WORKSPACE
    # dq aliasing q
    assert _status(lambda: f(h, *A[:3], W[0], W[1], A[3], A[4], A[0], A[6], A[7], W[2], W[3], WS, ws, 0)) == F.FMA_ERR_ARG
    # per-level plans validate the same way (their backward is built)
    pl = F.FMA(ndim=1, batch=1, heads=1, seq_len=4096, block=64, norm=F.FMA_NORM_PER_LEVEL)
    wsl = pl.backward_workspace_bytes
    assert _status(lambda: f(pl.handle, *A[:3], W[0], W[1], A[3], A[4], *A[5:], W[2], W[3], WS, wsl - 1, 0)) == \
        F.FMA_ERR_WORKSPACE
    assert _status(lambda: f(pl.handle, *A[:3], W[0], W[1], A[3], A[4], *A[5:], None, W[3], WS, wsl, 0)) == \
        F.FMA_ERR_NULL


def test_destroy_null_is_noop():
    F.fma_destroy(None)


def test_product_path_has_no_cpu_fallback(monkeypatch):
    """Without the built library the binding raises instead of computing."""
    monkeypatch.setattr(F, "_lib", None)
    monkeypatch.setattr(F, "LIB_PATH", "/nonexistent/libfma_mi355x.so")
    with pytest.raises(RuntimeError):
        F.FMA(ndim=1, batch=1, heads=1, seq_len=1024, block=64)


def test_product_does_not_import_oracle():
    import paper_2310_11960_amd
    import inspect
    src = inspect.getsource(paper_2310_11960_amd)
    assert "import oracle" not in src and "from oracle" not in src


def test_static_forward_rejects_large_plans_before_the_device():
    """fma_forward_static refuses a plan whose workspace exceeds its 32 MiB
    static buffer before any HIP call (fake pointers are never touched)."""
    op = F.FMA(ndim=1, batch=8, heads=16, seq_len=65536, block=128)
    assert op.workspace_bytes > 32 << 20
    fake = 1 << 20
    assert _status(lambda: F.fma_forward_static(op.handle, fake, fake, fake, fake, fake, fake, 0)) == \
        F.FMA_ERR_WORKSPACE
    assert "static scratch buffer holds" in F.fma_last_error()
    lin = F.FMA(ndim=1, batch=1, heads=1, seq_len=1024, block=64, linear=True)
    assert _status(lambda: F.fma_forward_static(lin.handle, fake, fake, fake, fake, fake, fake, 0)) == F.FMA_ERR_ARG
    assert _status(lambda: F.fma_forward_static(None, fake, fake, fake, fake, fake, fake, 0)) == F.FMA_ERR_NULL
