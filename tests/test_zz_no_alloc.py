"""fma_forward_static (the allocation-free forward: its workspace is the
library's static per-GPU buffer) against fma_forward_1d / fma_forward_2d with
a caller workspace, through the C ABI.  Same kernels, so the outputs must be
bitwise equal; two calls in a row, the second with a smaller input, check
that nothing depends on what the previous call left in the shared buffer."""
import numpy as np
import pytest
import torch

import fma_inputs
import oracle
import paper_2310_11960_amd as F

pytestmark = pytest.mark.gpu


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def _plan(w):
    return F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block, causal=w.causal,
                 dtype=w.torch_dtype, side=w.side, rank=w.rank)


def _both(w, dev):
    q, k, v, wk, wv = [t.to(dev) for t in fma_inputs.make_inputs(w)]
    op = _plan(w)
    ref = op.forward(q, k, v, wk, wv)                  # caller workspace
    out = torch.full_like(q, float("nan"))
    F.fma_forward_static(op.handle, q, k, v, wk, wv, out)   # static buffer
    torch.cuda.synchronize()
    return ref.cpu(), out.cpu(), (q, k, v, wk, wv)


@pytest.mark.parametrize("first,second", [
    ("C4", "small_causal"),
    ("C5", "small_2d"),
    ("C3_p4", "small_bidi_f32"),
])
def test_static_forward_matches_workspace_forward(first, second):
    dev = _dev()
    small = {
        "small_causal": fma_inputs.custom("small_causal", 1, True, "bf16", 1, 3, n=64 * 21, block=64, seed=3),
        "small_2d": fma_inputs.custom("small_2d", 2, False, "bf16", 2, 2, side=40, block=8, seed=4),
        "small_bidi_f32": fma_inputs.custom("small_bidi_f32", 1, False, "f32", 1, 2, n=1024, block=64, seed=5),
    }
    base, _, p = first.partition("_p")
    w1 = fma_inputs.WORKLOADS[base]
    if p:
        w1 = fma_inputs.with_rank(w1, int(p))
    w2 = small[second]
    assert _plan(w1).workspace_bytes > _plan(w2).workspace_bytes
    for w in (w1, w2):
        ref, out, (q, k, v, wk, wv) = _both(w, dev)
        assert torch.equal(out, ref), w.name
        # and the second, smaller call against the oracle on one slice
        if w is w2:
            b, h = w.batch - 1, w.heads - 1
            f = lambda t: t[b, h].double().cpu().numpy()   # noqa: E731
            if w.ndim == 1:
                o = oracle.forward_1d(f(q), f(k), f(v), w.block, wk[h].double().cpu().numpy(),
                                      wv[h].double().cpu().numpy(), causal=w.causal)
            else:
                o = oracle.forward_2d(f(q), f(k), f(v), w.side, w.block, wk[h].double().cpu().numpy(),
                                      wv[h].double().cpu().numpy())
            tol = 1e-5 if w.dtype == "f32" else 2e-2
            assert np.abs(out[b, h].double().numpy() - o).max() / np.abs(o).max() <= tol


def test_static_forward_repeated_calls_bitwise_equal():
    dev = _dev()
    w = fma_inputs.custom("rep", 1, False, "bf16", 2, 4, n=8192, block=128, seed=9)
    q, k, v, wk, wv = [t.to(dev) for t in fma_inputs.make_inputs(w)]
    op = _plan(w)
    a = op.forward_static(q, k, v, wk, wv)
    b = op.forward_static(q, k, v, wk, wv)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_static_forward_rejects_plans_beyond_the_buffer():
    dev = _dev()
    w = fma_inputs.custom("big", 1, False, "bf16", 8, 16, n=65536, block=128, seed=1)
    op = _plan(w)
    assert op.workspace_bytes > 32 << 20
    x = torch.empty(16, dtype=torch.bfloat16, device=dev)
    with pytest.raises(F.FmaError) as e:
        F.fma_forward_static(op.handle, x, x, x, x, x, x)
    assert e.value.status == F.FMA_ERR_WORKSPACE
    assert "static scratch buffer holds" in str(e.value)
