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
               side=w.side, linear=True)
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
        ref = oracle.forward_2d(_np(q), _np(k), _np(v), w.side, w.block, pk, pv, piq=pq)
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
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_linear_parity_small(case):
    name, ndim, dt, B, H, size, r = case
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, False, dt, B, H, n=size, block=r, seed=seed)
    else:
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size, block=r, seed=seed)
    _run_and_check(w)


@pytest.mark.parametrize("name", ["C4", "C5"])
def test_linear_parity_workloads(name):
    """Full-size launch (as the benchmark times it), every slice."""
    _run_and_check(fma_inputs.WORKLOADS[name], name + "_linear")
