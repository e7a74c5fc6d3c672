"""GPU parity of FMA-linear (fma_forward_linear: queries downsampled on every
coarse level, the coarse query of a token's own group scoring its far field)
against the fp64 oracle with the same query weights.  Tolerances as for the
forward: 1e-5 (fp32) and 2e-2 (bf16) relative per (batch, head) slice."""
import zlib

import numpy as np
import pytest
import torch

import fma_inputs
import oracle
import paper_2310_11960_amd as F
import parity_record

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def _np(t):
    return t.detach().to("cpu", torch.float64).numpy()


def rel_err(got, ref):
    return float(np.abs(got - ref).max() / max(np.abs(ref).max(), 1e-30))


def _run_and_check(w, case=None):
    """Every (batch, head) slice against the oracle (one call over the batch)."""
    dev = _dev()
    q, k, v, wk, wv = fma_inputs.make_inputs(w)
    wq = fma_inputs.make_query_weights(w)
    op = F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block, dtype=w.torch_dtype,
               side=w.side, linear=True, head_dim=w.head_dim)
    out = op.forward_linear(*[x.to(dev) for x in (q, k, v, wq, wk, wv)])
    torch.cuda.synchronize()
    out = out.cpu()
    assert torch.isfinite(out.float()).all()
    pk = None if wk.numel() == 0 else _np(wk)
    pv = None if wv.numel() == 0 else _np(wv)
    pq = None if wq.numel() == 0 else _np(wq)
    if w.ndim == 1:
        ref = oracle.forward_1d(_np(q), _np(k), _np(v), w.block, pk, pv, piq=pq)
    else:
        ref = oracle.forward_2d(_np(q), _np(k), _np(v), w.side, w.block, pk, pv, piq=pq, H=w.rows)
    got = _np(out)
    worst = worst_rms = 0.0
    bad = []
    for b in range(w.batch):
        for h in range(w.heads):
            e, er = parity_record.slice_errors(got[b, h], ref[b, h])
            worst, worst_rms = max(worst, e), max(worst_rms, er)
            if not e <= TOL[w.dtype]:
                bad.append((b, h, e))
    parity_record.record(case or w.name, "out", worst, worst_rms, TOL[w.dtype], w.batch * w.heads)
    print("%s worst slice rel err %.3e" % (case or w.name, worst), flush=True)
    assert not bad, (w.name, bad[:8])


CASES = [
    ("lin_bidi_f32_r64", 1, "f32", 1, 2, 1024, 64),
    ("lin_bidi_bf16_r128", 1, "bf16", 2, 2, 4096, 128),
    ("lin_ragged_bf16", 1, "bf16", 1, 3, 64 * 23, 64),
    ("lin_r256_bf16", 1, "bf16", 1, 1, 256 * 8, 256),
    ("lin_single_block", 1, "bf16", 1, 2, 64, 64),
    ("lin_2d_r8_bf16", 2, "bf16", 2, 2, 64, 8),
    ("lin_2d_r8_f32", 2, "f32", 1, 2, 32, 8),
    ("lin_2d_r16_bf16", 2, "bf16", 1, 2, 64, 16),
    ("lin_2d_ragged_f32", 2, "f32", 1, 1, 40, 8),
    ("lin_r16_bf16", 1, "bf16", 1, 2, 2048, 16),
    ("lin_r32_ragged_f32", 1, "f32", 1, 2, 32 * 23, 32),
    ("lin_2d_r4_bf16", 2, "bf16", 1, 2, 64, 4),
    ("lin_rect_wide_bf16", 2, "bf16", 1, 2, (32, 64), 8),
    ("lin_rect_ragged_f32", 2, "f32", 1, 1, (24, 40), 8),
    ("lin_rect_r4_bf16", 2, "bf16", 1, 2, (16, 48), 4),
]
# head dims 32 and 128 (the register-staged kernel's FMA-linear path)
HEADDIM_CASES = [
    ("lin_d128_bf16_r64", 1, "bf16", 1, 2, 1024, 64, 128),
    ("lin_d32_f32_r128", 1, "f32", 1, 2, 2048, 128, 32),
    ("lin_d128_2d_r8_bf16", 2, "bf16", 1, 2, 64, 8, 128),
]


@pytest.mark.parametrize("case", HEADDIM_CASES, ids=[c[0] for c in HEADDIM_CASES])
def test_linear_parity_head_dims(case):
    name, ndim, dt, B, H, size, r, d = case
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, False, dt, B, H, n=size, block=r, seed=seed, head_dim=d)
    else:
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size, block=r, seed=seed, head_dim=d)
    _run_and_check(w)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_linear_parity_small(case):
    name, ndim, dt, B, H, size, r = case
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, False, dt, B, H, n=size, block=r, seed=seed)
    elif isinstance(size, tuple):   # (rows, columns)
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size[1], height=size[0], block=r, seed=seed)
    else:
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size, block=r, seed=seed)
    _run_and_check(w)


@pytest.mark.parametrize("name", ["C4", "C5"])
def test_linear_parity_workloads(name):
    """Full-size launch (as the benchmark times it), every slice."""
    _run_and_check(fma_inputs.WORKLOADS[name], name + "_linear")


# ------------------------------------------------------------ backward
NAMES = ["dq", "dk", "dv", "dwk", "dwv", "dwq"]


def _backward_and_check(w, case, slices=None, whead=None):
    """fma_backward_linear against the oracle's FMA-linear gradients: dq, dk,
    dv per (batch, head) slice (every slice, or `slices`), and the three
    weight gradients per head (the oracle's per-slice gradients summed over
    the batch; every head, or head `whead`)."""
    dev = _dev()
    q, k, v, wk, wv = fma_inputs.make_inputs(w)
    wq = fma_inputs.make_query_weights(w)
    g = torch.Generator().manual_seed(zlib.crc32(case.encode()) % 1000 + 1)
    dout = torch.randn(q.shape, generator=g).to(q.dtype)
    op = F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block, dtype=w.torch_dtype,
               side=w.side, linear=True, head_dim=w.head_dim)
    t = [x.to(dev) for x in (q, k, v, wk, wv, wq, dout)]
    out = op.forward_linear(t[0], t[1], t[2], t[5], t[3], t[4])
    grads = op.backward_linear(t[0], t[1], t[2], t[3], t[4], t[5], out, t[6])
    torch.cuda.synchronize()
    grads = [None if x is None else x.cpu() for x in grads]
    slices = slices or [(b, h) for b in range(w.batch) for h in range(w.heads)]
    heads = [whead] if whead is not None else list(range(w.heads))
    refs = {}

    def ref_of(b, h):
        if (b, h) not in refs:
            pk = None if wk.numel() == 0 else _np(wk[h])
            pv = None if wv.numel() == 0 else _np(wv[h])
            pq = None if wq.numel() == 0 else _np(wq[h])
            if w.ndim == 1:
                refs[(b, h)] = oracle.backward_1d(_np(q[b, h]), _np(k[b, h]), _np(v[b, h]), w.block, pk, pv,
                                                  _np(dout[b, h]), piq=pq if pq is not None else np.zeros(0))
            else:
                refs[(b, h)] = oracle.backward_2d(_np(q[b, h]), _np(k[b, h]), _np(v[b, h]), w.side, w.block, pk,
                                                  pv, _np(dout[b, h]), piq=pq if pq is not None else np.zeros(0),
                                                  H=w.rows)
        return refs[(b, h)]

    bad = []
    for x in range(3):
        errs = [parity_record.slice_errors(_np(grads[x][b, h]), ref_of(b, h)[x]) for (b, h) in slices]
        worst = max(e[0] for e in errs)
        parity_record.record(case, NAMES[x], worst, max(e[1] for e in errs), TOL[w.dtype], len(slices))
        if not worst <= TOL[w.dtype]:
            bad.append((NAMES[x], worst))
    if grads[3] is not None:
        for x in (3, 4, 5):
            errs = []
            for h in heads:
                acc = sum(ref_of(b, h)[x] for b in range(w.batch))
                errs.append(parity_record.slice_errors(_np(grads[x][h]), acc))
            worst = max(e[0] for e in errs)
            parity_record.record(case, NAMES[x], worst, max(e[1] for e in errs), TOL[w.dtype], len(heads))
            if not worst <= TOL[w.dtype]:
                bad.append((NAMES[x], worst))
    print(case, "backward", bad or "ok", flush=True)
    assert not bad, (case, bad)


BWD_CASES = [
    ("lin_bwd_f32_r64", 1, "f32", 1, 2, 512, 64),
    ("lin_bwd_bf16_r128", 1, "bf16", 2, 2, 2048, 128),
    ("lin_bwd_ragged_bf16", 1, "bf16", 1, 2, 64 * 11, 64),
    ("lin_bwd_r256_bf16", 1, "bf16", 1, 1, 256 * 8, 256),
    ("lin_bwd_single_block", 1, "bf16", 1, 2, 64, 64),
    ("lin_bwd_2d_r8_bf16", 2, "bf16", 1, 2, 64, 8),
    ("lin_bwd_2d_r8_f32", 2, "f32", 1, 1, 32, 8),
    ("lin_bwd_2d_ragged_f32", 2, "f32", 1, 1, 40, 8),
    ("lin_bwd_2d_r16_bf16", 2, "bf16", 1, 1, 64, 16),
    ("lin_bwd_r16_bf16", 1, "bf16", 1, 2, 1024, 16),
    ("lin_bwd_2d_r4_f32", 2, "f32", 1, 1, 32, 4),
    ("lin_bwd_rect_tall_bf16", 2, "bf16", 1, 2, (64, 24), 8),
    ("lin_bwd_rect_ragged_f32", 2, "f32", 1, 1, (40, 24), 8),
]


@pytest.mark.parametrize("case", BWD_CASES, ids=[c[0] for c in BWD_CASES])
def test_linear_backward_small(case):
    name, ndim, dt, B, H, size, r = case
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, False, dt, B, H, n=size, block=r, seed=seed)
    elif isinstance(size, tuple):   # (rows, columns)
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size[1], height=size[0], block=r, seed=seed)
    else:
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size, block=r, seed=seed)
    _backward_and_check(w, name)


@pytest.mark.parametrize("name,slices,whead", [("C4", [(0, 0), (1, 15)], 15), ("C5", [(0, 0), (15, 7)], 7)])
def test_linear_backward_workloads(name, slices, whead):
    """Full-size launch: the first and the last slice, and one head's weights."""
    _backward_and_check(fma_inputs.WORKLOADS[name], name + "_linear_bwd", slices, whead)
