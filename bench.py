"""Benchmark of the FMA forward pass on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload C4]

A step is one full forward pass (coarsening + fused multilevel attention)
over one batch of the workload, inputs resident in HBM.  The headline
workload is the 1D bidirectional long-context shape (B=2, H=16, n=65536,
d=64, r=128, bf16); the other long-sequence shapes (causal LM n=16384, 2D
128x128 map), and all three with coarse level rank 4 (four basis vectors per
level, the paper's experimental setting; names ending in _p4), C4 and C5
under the printed per-level normalisation (names ending in _level) and as
FMA-linear (queries downsampled on every coarse level; _linear), are timed in
the same run and reported under "others".

Prints ONE JSON line.  `value` is tokens per second of the whole forward
call, timed by the wall clock over --steps calls after --warmup calls;
`event_ms_per_step` is the same steps timed with HIP events recorded before
every step (first_step_ms / last_step_ms show the GPU's clock ramp after the
warm-up).  The backward pass (fma_backward) of C4, C3 and C5, and of C4
under the per-level normalisation and as FMA-linear (fma_backward_linear), is
timed after the forward workloads and reported under "backward" (not part of
`value`).
Per-kernel averages come from HIP events recorded on the stream the kernels
run on, around the two kernels of the same number of steps run once more.
The roofline entry is for the fused attention kernel: algorithmic flops
(4 * d per query-source pair) per launch over its average duration, against
the bf16 dense MFMA peak.  The CPU baseline is the fp64 oracle on distinct
(batch, head) slices of the benchmarked inputs, as many as fit in ~12 s,
each also compared with the GPU's output of that slice.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "FMA fwd tokens/s/GPU at n=16K–64K; % bf16 MFMA peak; coarsen HBM GB/s"
PEAK_BF16_TFLOPS = 2500.0
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
D = 64


# ------------------------------------------------------------ measured traffic
# HBM bytes per launch from two rocprofv3 counter passes (FETCH_SIZE, then
# WRITE_SIZE), each scaled by what the same counter reads for a plain device
# copy of known size.  The figures are stored with a digest of the sources
# that determine the kernels and their launch shapes; once any of them
# changes, the stored traffic no longer describes the kernel and is not
# reported.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
_COMMON_SOURCES = ["paper_2310_11960_amd/csrc/fma_api.hip", "paper_2310_11960_amd/csrc/fma_device.hpp",
                   "paper_2310_11960_amd/csrc/fma_kernels.hpp", "paper_2310_11960_amd/build.py"]
KERNEL_SOURCES = {
    "attend": ["paper_2310_11960_amd/csrc/attend_mfma.hip", "paper_2310_11960_amd/csrc/attend.hip"] + _COMMON_SOURCES,
    "coarsen": ["paper_2310_11960_amd/csrc/coarsen.hip"] + _COMMON_SOURCES,
}


def sources_digest(kind):
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[kind]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload, kind):
    """Counter-measured HBM bytes per launch of one pass, or None."""
    try:
        with open(TRAFFIC_FILE) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    e = d.get("kernels", {}).get("%s|%s" % (workload, kind))
    if not e or e.get("sources_sha256") != sources_digest(kind):
        return None
    return e.get("bytes_per_launch")


# ------------------------------------------------------------ work model
def _levels(ratio):
    L, p = 0, 1
    while p < ratio:
        p, L = 2 * p, L + 1
    return L


def workload(fma_inputs, name):
    """A named workload; NAME_pP is workload NAME with rank P (a trailing
    _level selects the normalisation, see per_level; _linear FMA-linear)."""
    base, _, p = name.replace("_level", "").replace("_linear", "").partition("_p")
    w = fma_inputs.WORKLOADS[base]
    return fma_inputs.with_rank(w, int(p)) if p else w


def per_level(name):
    """NAME_level: the printed per-level normalisation instead of the joint one."""
    return name.endswith("_level")


def linear(name):
    """NAME_linear: FMA-linear (queries downsampled on every coarse level)."""
    return name.endswith("_linear")


def work_model(w):
    """Algorithmic work of one forward over the whole batch (n / r a power of
    two, as in every benchmark workload).

    sources : query-source pairs (near tokens + far groups), from the
              closed-form counts of the near window and the 3 (causal: 1.5 on
              average) groups per level and query; 2D: 3x3 cells and 27
              squares per level, clipped at the map edges.  At rank p every
              far group is p sources, and there are p times the coarse rows
              and weights.
    flops   : 4 * d per pair (q.k and p*v, multiply + add each).
    bytes   : Q, K, V, O once + K_bar, V_bar once (fused kernel);
              K, V read + K_bar, V_bar written + weights (coarsening).
    """
    S = w.batch * w.heads
    esz = 2 if w.dtype == "bf16" else 4
    r = w.block
    if w.ndim == 1:
        n = w.n
        L = _levels(n // r)
        if w.causal:
            near = r * (n - r) + n * (r + 1) // 2
            far = (3 * n * (L - 2) + 6 * r) // 2 if L >= 2 else 0
        else:
            near = r * (3 * n - 2 * r)
            far = 3 * n * (L - 2) + 6 * r if L >= 2 else 0
        R = sum(-(-n // (r << l)) for l in range(L - 1))
        wlen = sum(r << l for l in range(L - 1))
    else:
        W = w.side
        M0 = W // r
        L = _levels(M0)
        near = r ** 4 * (3 * M0 - 2) ** 2
        far = 0
        R = 0
        for l in range(1, L):
            s = r * 2 ** (l - 1)
            M = W // s
            far += s * s * ((6 * M - 8) ** 2 - (3 * M - 2) ** 2)
            R += M * M
        wlen = sum(2 * (r << l) for l in range(L - 1))
        n = W * W
    far, R, wlen = far * w.rank, R * w.rank, wlen * w.rank
    pairs = S * (near + far)
    flops = 4 * D * pairs
    fused_bytes = S * (4 * n * D * esz + 2 * R * D * esz)
    coarsen_bytes = S * (2 * n * D * esz + 2 * R * D * esz) + 2 * w.heads * wlen * 4
    return dict(pairs=pairs, flops=flops, fused_bytes=fused_bytes, coarsen_bytes=coarsen_bytes,
                tokens=w.batch * n, R=R)


# ------------------------------------------------------------ timing
def _time_events(torch, fn, iters):
    """Average milliseconds of fn() over iters launches, HIP events on the
    current stream (the stream the library launches on)."""
    st = torch.cuda.current_stream()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record(st)
    for _ in range(iters):
        fn()
    b.record(st)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / iters


def bench_workload(torch, F, fma_inputs, name, steps, warmup, dense=False, cpu_budget_s=0.0):
    w = workload(fma_inputs, name)
    dev = torch.device("cuda:0")
    q, k, v, wk, wv = fma_inputs.make_inputs(w, device=dev)
    op = F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block,
               causal=w.causal, dtype=w.torch_dtype, side=w.side, rank=w.rank,
               norm=F.FMA_NORM_PER_LEVEL if per_level(name) else F.FMA_NORM_JOINT, linear=linear(name))
    ws = op.new_workspace(dev)
    out = torch.empty_like(q)
    wq = fma_inputs.make_query_weights(w, device=dev) if linear(name) else None

    def step():
        if wq is not None:
            op.forward_linear(q, k, v, wq, wk, wv, out=out, workspace=ws)
        else:
            op.forward(q, k, v, wk, wv, out=out, workspace=ws)

    for _ in range(warmup):
        step()
    # The timed steps: wall clock between two synchronisations, and a HIP event
    # before every step on the stream the library launches on (the events add
    # no GPU work), so that the event time covers exactly the same steps.
    st = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        evs[i].record(st)
        step()
    evs[steps].record(st)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / steps
    per_step = [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]
    timed = dict(ms_per_step=wall_ms, event_ms_per_step=sum(per_step) / steps,
                 first_step_ms=per_step[0], last_step_ms=per_step[-1],
                 tokens_per_s=work_model(w)["tokens"] / (wall_ms * 1e-3))
    if wq is not None:
        # FMA-linear: the whole call only (two coarsening passes, then attention)
        res = dict(workload=name, note=w.note, rank=w.rank, norm="joint", variant="FMA-linear", **timed)
        del q, k, v, out, ws, wq
        torch.cuda.empty_cache()
        return res, w

    # Per-kernel averages: the same steps again, split at the kernel boundary
    # (coarsening, then attention, exactly what the forward call launches),
    # with HIP events on the stream the library launches on.  Every attention
    # launch in the run therefore follows a coarsening pass, as in the
    # forward call, so a profiler's average over all launches sees the same
    # population.
    st = torch.cuda.current_stream()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for e in evs:
        e[0].record(st)
        op.coarsen(k, v, wk, wv, workspace=ws)
        e[1].record(st)
        op.attend(q, k, v, ws, out=out)
        e[2].record(st)
    torch.cuda.synchronize()
    coarsen_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / steps
    attend_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / steps
    step_ms = sum(e[0].elapsed_time(e[2]) for e in evs) / steps
    wm = work_model(w)
    res = dict(
        workload=name, note=w.note, rank=w.rank, norm="per_level" if per_level(name) else "joint",
        **timed, split_event_ms_per_step=step_ms,
        attend_us=attend_ms * 1e3, coarsen_us=coarsen_ms * 1e3,
        attend_tflops=wm["flops"] / (attend_ms * 1e-3) / 1e12,
        attend_gbs=wm["fused_bytes"] / (attend_ms * 1e-3) / 1e9,
        coarsen_gbs=wm["coarsen_bytes"] / (coarsen_ms * 1e-3) / 1e9,
        flops_per_launch=wm["flops"], fused_bytes_per_launch=wm["fused_bytes"],
        coarsen_bytes_per_launch=wm["coarsen_bytes"], pairs=wm["pairs"],
        attend_traffic_bytes=measured_traffic(name, "attend"),
        coarsen_traffic_bytes=measured_traffic(name, "coarsen"),
    )
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    ai = wm["flops"] / wm["fused_bytes"]
    res["attend_frac_mfma_peak"] = res["attend_tflops"] / peak
    res["attend_roofline_tflops"] = min(peak, ai * PEAK_HBM_GBS / 1e3)
    res["attend_frac_roofline"] = res["attend_tflops"] / res["attend_roofline_tflops"]
    res["coarsen_frac_hbm"] = res["coarsen_gbs"] / PEAK_HBM_GBS
    if cpu_budget_s:
        res["cpu_baseline"] = cpu_baseline(torch, w, q, k, v, wk, wv, out, cpu_budget_s)
    if dense:
        it = 3
        dense_ms = _time_events(torch, lambda: op.dense_reference(q, k, v, out=out), it)
        pairs = w.batch * w.heads * (w.n * (w.n + 1) // 2 if w.causal else w.n * w.n)
        res["dense_ms"] = dense_ms
        res["dense_tflops"] = 4 * D * pairs / (dense_ms * 1e-3) / 1e12
        res["fma_speedup_vs_dense"] = dense_ms / wall_ms
    del q, k, v, out, ws
    torch.cuda.empty_cache()
    return res, w


def bench_sweep(torch, F, fma_inputs, ns, causal, heads=16, block=128):
    """FMA's whole forward call against this library's dense HIP attention
    (fma_dense_reference) over sequence lengths ns, bf16, one sequence of
    `heads` heads (d = 64, r = 128): the paper's efficiency comparison with
    sequence length (Sec. 4), on synthetic inputs.  HIP events, 20 FMA calls
    after 5 warm-ups and 3 dense calls after one."""
    dev = torch.device("cuda:0")
    rows = []
    for n in ns:
        w = fma_inputs.custom("sweep", 1, causal, "bf16", 1, heads, n=n, block=block, seed=2310 + n % 997)
        q, k, v, wk, wv = fma_inputs.make_inputs(w, device=dev)
        op = F.FMA(ndim=1, batch=1, heads=heads, seq_len=n, block=block, causal=causal, dtype=w.torch_dtype)
        ws = op.new_workspace(dev)
        out = torch.empty_like(q)
        fwd = lambda: op.forward(q, k, v, wk, wv, out=out, workspace=ws)   # noqa: E731
        for _ in range(5):
            fwd()
        fma_ms = _time_events(torch, fwd, 20)
        dense = lambda: op.dense_reference(q, k, v, out=out)   # noqa: E731
        dense()
        dense_ms = _time_events(torch, dense, 3)
        rows.append({"n": n, "causal": causal, "fma_ms": fma_ms, "dense_ms": dense_ms,
                     "speedup": dense_ms / fma_ms, "fma_tokens_per_s": n / (fma_ms * 1e-3),
                     "fma_workspace_bytes": op.workspace_bytes})
        print("sweep n=%d causal=%d fma %.3f ms dense %.3f ms" % (n, causal, fma_ms, dense_ms),
              file=sys.stderr, flush=True)
        del q, k, v, out, ws
        torch.cuda.empty_cache()
    return rows


def bench_backward(torch, F, fma_inputs, name, steps=5, warmup=2):
    """fma_backward (gradients of sum(dO * O) for Q, K, V and both weight
    sets; NAME_level: the per-level normalisation; NAME_linear:
    fma_backward_linear, with the query weights' gradient too) on the
    workload, HIP events on the library's stream.  Algorithmic work: 10 * d
    flop per (query, source) pair (recomputed scores, dP, dQ, dK, dV), the
    usual accounting for attention backward."""
    w = workload(fma_inputs, name)
    linear = name.endswith("_linear")
    dev = torch.device("cuda:0")
    q, k, v, wk, wv = fma_inputs.make_inputs(w, device=dev)
    op = F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block,
               causal=w.causal, dtype=w.torch_dtype, side=w.side, rank=w.rank,
               norm=F.FMA_NORM_PER_LEVEL if per_level(name) else F.FMA_NORM_JOINT, linear=linear)
    g = torch.Generator(device=dev)
    g.manual_seed(w.seed + 7)
    dout = torch.randn(q.shape, generator=g, device=dev).to(q.dtype)
    ws = torch.empty(op.backward_workspace_bytes, dtype=torch.uint8, device=dev)
    if linear:
        wq = fma_inputs.make_query_weights(w, device=dev)
        out = op.forward_linear(q, k, v, wq, wk, wv)

        def step():
            op.backward_linear(q, k, v, wk, wv, wq, out, dout, workspace=ws)
    else:
        out = op.forward(q, k, v, wk, wv)

        def step():
            op.backward(q, k, v, wk, wv, out, dout, workspace=ws)

    for _ in range(warmup):
        step()
    ms = _time_events(torch, step, steps)
    wm = work_model(w)
    tf = 10 * D * wm["pairs"] / (ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    del q, k, v, out, dout, ws
    torch.cuda.empty_cache()
    return {"workload": name, "ms": ms, "tokens_per_s": wm["tokens"] / (ms * 1e-3),
            "tflops_alg": tf, "frac_mfma_peak": tf / peak,
            "workspace_bytes": op.backward_workspace_bytes}


def copy_reference(torch, nbytes=1 << 30, iters=10):
    """Achievable HBM rate: a plain device-to-device copy of nbytes (read +
    write = 2 * nbytes per launch), also the calibration kernel for the
    FETCH_SIZE / WRITE_SIZE counters."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    src.fill_(1)
    for _ in range(2):
        dst.copy_(src)
    ms = _time_events(torch, lambda: dst.copy_(src), iters)
    del src, dst
    torch.cuda.empty_cache()
    return {"bytes_per_launch": 2 * nbytes, "avg_us": ms * 1e3, "gbs": 2 * nbytes / (ms * 1e-3) / 1e9}


def read_stream_reference(torch, F, nbytes=1 << 30, write_every=64, iters=20):
    """Achievable rate of the coarsening's traffic mix: the library's
    fma_stream_reference kernel reads nbytes once with 16-byte loads and
    writes one 16-byte word per write_every words read (the coarsening writes
    1/40 to 1/60 of what it reads).  Bytes = read + written."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    src.fill_(1)
    nchunk = -(-nbytes // 32768)
    dst_bytes = nchunk * (2048 // write_every) * 16
    dst = torch.empty(dst_bytes, dtype=torch.uint8, device="cuda:0")

    def run():
        F.fma_stream_reference(src, nbytes, dst, dst_bytes, write_every)

    for _ in range(3):
        run()
    ms = _time_events(torch, run, iters)
    del src, dst
    torch.cuda.empty_cache()
    moved = nbytes + dst_bytes
    return {"kernel": "stream_ref_kernel (fma_stream_reference)", "read_bytes": nbytes, "write_bytes": dst_bytes,
            "avg_us": ms * 1e3, "gbs": moved / (ms * 1e-3) / 1e9}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(torch, w, q, k, v, wk, wv, out, budget_s=12.0):
    """The fp64 oracle on distinct (batch, head) slices of the benchmarked
    inputs (copied from the GPU), in slice order, as many as fit in about
    budget_s seconds (at least one), on the host's cores.  Each slice is also
    compared with the GPU output of the same slice (inf-norm and RMS relative
    error).  Then a per-core figure: the same oracle on one thread, on the
    first slice of the small 1D workloads (fp32 n=1024 and bf16 causal
    n=4096)."""
    import ctypes

    import numpy as np

    import fma_inputs
    import oracle

    oracle.num_levels(2)          # build / load outside the timed region
    f64 = lambda t: t.detach().to("cpu", torch.float64).numpy()   # noqa: E731
    done, t, worst, worst_rms = 0, 0.0, 0.0, 0.0
    for b in range(w.batch):
        for h in range(w.heads):
            qs, ks, vs = f64(q[b, h]), f64(k[b, h]), f64(v[b, h])
            pk, pv = f64(wk[h]), f64(wv[h])
            t0 = time.perf_counter()
            if w.ndim == 1:
                ref = oracle.forward_1d(qs, ks, vs, w.block, pk, pv, causal=w.causal, rank=w.rank)
            else:
                ref = oracle.forward_2d(qs, ks, vs, w.side, w.block, pk, pv, rank=w.rank)
            t += time.perf_counter() - t0
            done += 1
            d = f64(out[b, h]) - ref
            worst = max(worst, float(np.abs(d).max() / np.abs(ref).max()))
            worst_rms = max(worst_rms, float(np.sqrt((d ** 2).mean() / (ref ** 2).mean())))
            if t >= budget_s:
                break
        if t >= budget_s:
            break
    cores = int(os.environ.get("OMP_NUM_THREADS") or len(os.sched_getaffinity(0)))

    # one thread: the per-core figure
    per_core = {}
    try:
        gomp = ctypes.CDLL("libgomp.so.1")
        prev = gomp.omp_get_max_threads()
        gomp.omp_set_num_threads(1)
        try:
            for name in ("C1", "C2"):
                sw = fma_inputs.WORKLOADS[name]
                one = fma_inputs.Workload(**{**sw.__dict__, "batch": 1, "heads": 1})
                sq, sk, sv, swk, swv = fma_inputs.make_inputs(one)
                a = [x[0, 0].double().numpy() for x in (sq, sk, sv)]
                t0 = time.perf_counter()
                oracle.forward_1d(*a, sw.block, swk[0].double().numpy(), swv[0].double().numpy(), causal=sw.causal)
                per_core[name] = sw.n / (time.perf_counter() - t0)
        finally:
            gomp.omp_set_num_threads(prev)
    except OSError:
        pass
    return {"value": done * w.n / t, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu_model": _cpu_model(),
            "sample": "%d distinct (batch, head) slices of %s (the benchmarked inputs, n=%d each), fp64, %.1f s"
                      % (done, w.name, w.n, t),
            "parity_vs_gpu": {"slices": done, "max_rel": worst, "rms_rel": worst_rms},
            "per_core_tokens_per_s": {k_: round(v_, 1) for k_, v_ in per_core.items()}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="C4")
    ap.add_argument("--others", default="C3,C5,C4_p4,C3_p4,C5_p4,C4_level,C5_level,C4_linear,C5_linear")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-copy", action="store_true", help="skip the plain-copy HBM reference")
    ap.add_argument("--backward", default="C4,C3,C5,C4_level,C4_linear",
                    help="workloads whose backward pass is timed too (empty: none)")
    ap.add_argument("--sweep", default="",
                    help="sequence lengths (comma-separated) for an FMA-vs-dense forward sweep, "
                         "1D bf16, 16 heads, r = 128, bidirectional and causal (empty: none)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (--gpus %d requested)"
              % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    import fma_inputs
    import paper_2310_11960_amd as F
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    F.library()

    head, w = bench_workload(torch, F, fma_inputs, args.workload, args.steps, args.warmup,
                             dense=not args.no_dense, cpu_budget_s=0.0 if args.no_cpu_baseline else 12.0)
    others = {}
    for name in [x for x in args.others.split(",") if x and x != args.workload]:
        others[name], _ = bench_workload(torch, F, fma_inputs, name, args.steps, args.warmup,
                                         dense=not args.no_dense and "_" not in name)

    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    line = {
        "metric": METRIC,
        "value": head["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": "%s: %s; B=%d H=%d n=%d d=%d r=%d%s" % (
            w.name, w.note, w.batch, w.heads, w.n, w.head_dim, w.block,
            (" (%dx%d map)" % (w.side, w.side)) if w.ndim == 2 else ""),
            "global_batch": w.batch, "seq_len": w.n, "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "achieved": head["attend_tflops"], "peak": peak,
                     "unit": "TFLOP/s", "frac": head["attend_tflops"] / peak,
                     "traffic": measured_traffic(w.name, "attend"),
                     "kernel": "attend_mfma_kernel (fused multilevel attention, bf16)"
                     if w.dtype == "bf16" else "attend_kernel (fused multilevel attention, fp32)",
                     "flops_per_launch": head["flops_per_launch"],
                     "algorithmic_bytes_per_launch": head["fused_bytes_per_launch"],
                     "avg_launch_us": head["attend_us"]},
        "coarsen": {"bound": "hbm", "achieved": head["coarsen_gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": head["coarsen_frac_hbm"], "avg_us": head["coarsen_us"],
                    "bytes_per_launch": head["coarsen_bytes_per_launch"],
                    "traffic": measured_traffic(w.name, "coarsen")},
        "detail": head,
        "others": others,
    }
    if args.backward:
        line["backward"] = {name: bench_backward(torch, F, fma_inputs, name)
                            for name in args.backward.split(",") if name}
    if not args.no_copy:
        line["hbm_copy_reference"] = copy_reference(torch)
        ref = read_stream_reference(torch, F)
        ref["coarsen_frac_of_reference"] = head["coarsen_gbs"] / ref["gbs"]
        line["hbm_read_stream_reference"] = ref
        line["coarsen"]["frac_of_read_stream_reference"] = ref["coarsen_frac_of_reference"]
    if args.sweep:
        ns = [int(x) for x in args.sweep.split(",") if x]
        line["sweep"] = bench_sweep(torch, F, fma_inputs, ns, False) + bench_sweep(torch, F, fma_inputs, ns, True)
    if "cpu_baseline" in head:
        line["cpu_baseline"] = head.pop("cpu_baseline")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
