"""GPU parity of the backward pass (fma_backward, through the C ABI) against
the fp64 oracle's gradients on the same seeded inputs.

Tolerance per (batch, head) slice and tensor: max|g_gpu - g_ref| / max|g_ref|
<= 1e-5 for fp32 and 2e-2 for bf16 I/O (fp32 accumulation; bf16 runs round
P and dS to bf16 for the matrix cores and store the gradients in bf16).
Weight gradients are compared per head over the whole vector.  The oracle
receives the GPU forward's own output O only through dO . O, which the
backward takes as given, so the reference uses the oracle's forward.
"""
import zlib

import numpy as np
import pytest
import torch

import fma_inputs
import oracle
import paper_2310_11960_amd as F

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


def _case(name, ndim, causal, dt, B, H, size, r, p=1, shared=False):
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, causal, dt, B, H, n=size, block=r, seed=seed, rank=p)
    else:
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size, block=r, seed=seed, rank=p)
    q, k, v, wk, wv = fma_inputs.make_inputs(w, weights_shared=shared)
    g = torch.Generator().manual_seed(seed + 1)
    dout = torch.randn(q.shape, generator=g).to(q.dtype)
    return w, q, k, v, wk, wv, dout


def _gpu_backward(w, q, k, v, wk, wv, dout, dev, shared=False):
    op = F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block, causal=w.causal,
               dtype=w.torch_dtype, side=w.side, weights_per_head=not shared, rank=w.rank)
    t = [x.to(dev) for x in (q, k, v, wk, wv, dout)]
    out = op.forward(*t[:5])
    grads = op.backward(t[0], t[1], t[2], t[3], t[4], out, t[5])
    torch.cuda.synchronize()
    return out.cpu(), [None if x is None else x.cpu() for x in grads]


def _oracle_grads(w, q, k, v, wk, wv, dout, b, h, shared=False):
    pk = None if wk.numel() == 0 else _np(wk if shared else wk[h])
    pv = None if wv.numel() == 0 else _np(wv if shared else wv[h])
    if w.ndim == 1:
        return oracle.backward_1d(_np(q[b, h]), _np(k[b, h]), _np(v[b, h]), w.block, pk, pv, _np(dout[b, h]),
                                  causal=w.causal, rank=w.rank)
    return oracle.backward_2d(_np(q[b, h]), _np(k[b, h]), _np(v[b, h]), w.side, w.block, pk, pv,
                              _np(dout[b, h]), rank=w.rank)


def _check(w, q, k, v, wk, wv, dout, grads, shared=False):
    worst = [0.0] * 5
    wref_k = wref_v = 0.0
    for b in range(w.batch):
        for h in range(w.heads):
            ref = _oracle_grads(w, q, k, v, wk, wv, dout, b, h, shared)
            for x in range(3):
                worst[x] = max(worst[x], rel_err(_np(grads[x][b, h]), ref[x]))
            if ref[3] is not None:
                wref_k = wref_k + ref[3]
                wref_v = wref_v + ref[4]
    if grads[3] is not None:
        # per-head weights: the oracle's per-slice gradients summed over the batch
        if shared:
            worst[3] = rel_err(_np(grads[3]), wref_k)
            worst[4] = rel_err(_np(grads[4]), wref_v)
        else:
            accs_k = [0.0] * w.heads
            accs_v = [0.0] * w.heads
            for b in range(w.batch):
                for h in range(w.heads):
                    ref = _oracle_grads(w, q, k, v, wk, wv, dout, b, h, shared)
                    accs_k[h] = accs_k[h] + ref[3]
                    accs_v[h] = accs_v[h] + ref[4]
            worst[3] = max(rel_err(_np(grads[3][h]), accs_k[h]) for h in range(w.heads))
            worst[4] = max(rel_err(_np(grads[4][h]), accs_v[h]) for h in range(w.heads))
    print("%s rel err dq %.2e dk %.2e dv %.2e dwk %.2e dwv %.2e" % (w.name, *worst), flush=True)
    for x, e in enumerate(worst):
        assert e <= TOL[w.dtype], (w.name, ["dq", "dk", "dv", "dwk", "dwv"][x], e)


CASES = [
    # name, ndim, causal, dtype, B, H, n/side, r, rank
    ("bwd_bidi_f32_r64", 1, False, "f32", 1, 2, 512, 64, 1),
    ("bwd_causal_f32_r64", 1, True, "f32", 1, 2, 512, 64, 1),
    ("bwd_bidi_bf16_r64", 1, False, "bf16", 2, 2, 1024, 64, 1),
    ("bwd_causal_bf16_r128", 1, True, "bf16", 1, 2, 2048, 128, 1),
    ("bwd_ragged_bidi_bf16", 1, False, "bf16", 1, 1, 64 * 11, 64, 1),
    ("bwd_p3_causal_f32", 1, True, "f32", 1, 1, 1024, 64, 3),
    ("bwd_p4_bidi_bf16", 1, False, "bf16", 1, 2, 2048, 64, 4),
    ("bwd_single_block_bf16", 1, True, "bf16", 1, 2, 64, 64, 1),
    # several query-pass workgroups per block: 2 (r=256 bf16, r=128 fp32), 3 (r=192 bf16)
    ("bwd_bidi_bf16_r256", 1, False, "bf16", 1, 2, 2048, 256, 1),
    ("bwd_causal_bf16_r192_p2", 1, True, "bf16", 1, 1, 1536, 192, 2),
    ("bwd_bidi_f32_r128", 1, False, "f32", 1, 1, 1024, 128, 1),
    ("bwd_2d_r8_f32", 2, False, "f32", 1, 1, 32, 8, 1),
    ("bwd_2d_r8_bf16", 2, False, "bf16", 1, 2, 64, 8, 1),
    ("bwd_2d_r16_bf16", 2, False, "bf16", 1, 1, 64, 16, 1),
    ("bwd_2d_ragged_bf16_p2", 2, False, "bf16", 1, 1, 40, 8, 2),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_backward_parity(case):
    dev = _dev()
    w, q, k, v, wk, wv, dout = _case(*case)
    _, grads = _gpu_backward(w, q, k, v, wk, wv, dout, dev)
    _check(w, q, k, v, wk, wv, dout, grads)


def test_backward_shared_weights():
    dev = _dev()
    w, q, k, v, wk, wv, dout = _case("bwd_shared", 1, True, "bf16", 2, 2, 1024, 64, 1, shared=True)
    _, grads = _gpu_backward(w, q, k, v, wk, wv, dout, dev, shared=True)
    _check(w, q, k, v, wk, wv, dout, grads, shared=True)


def test_backward_deterministic():
    dev = _dev()
    w, q, k, v, wk, wv, dout = _case("bwd_det", 1, False, "bf16", 1, 2, 2048, 128, 2)
    _, g1 = _gpu_backward(w, q, k, v, wk, wv, dout, dev)
    _, g2 = _gpu_backward(w, q, k, v, wk, wv, dout, dev)
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)


@pytest.mark.parametrize("name,slices", [("C3", [(0, 0), (7, 11)]), ("C5", [(0, 0)])])
def test_backward_workloads(name, slices):
    """Full-size launch; oracle on sampled slices (dq, dk, dv)."""
    dev = _dev()
    w = fma_inputs.WORKLOADS[name]
    q, k, v, wk, wv = fma_inputs.make_inputs(w)
    g = torch.Generator().manual_seed(7)
    dout = torch.randn(q.shape, generator=g).to(q.dtype)
    _, grads = _gpu_backward(w, q, k, v, wk, wv, dout, dev)
    for (b, h) in slices:
        ref = _oracle_grads(w, q, k, v, wk, wv, dout, b, h)
        for x in range(3):
            e = rel_err(_np(grads[x][b, h]), ref[x])
            print(name, b, h, ["dq", "dk", "dv"][x], "%.2e" % e, flush=True)
            assert e <= TOL[w.dtype], (name, b, h, x, e)
