"""The forward (with a caller workspace and allocation-free), the backward
and the FMA-linear forward captured in a HIP graph (torch.cuda.CUDAGraph) and
replayed.  The library allocates nothing and records no memset, so the
captured launches are replayable: every replay, with new inputs copied into
the captured buffers and eager library calls in between, must equal the
eager call on the same inputs bitwise (the kernels are deterministic)."""
import pytest
import torch

import fma_inputs
import paper_2310_11960_amd as F

pytestmark = pytest.mark.gpu

CASES = {
    "bidi_1d": dict(ndim=1, causal=False, dtype="bf16", batch=1, heads=4, n=4096, block=128),
    "causal_1d": dict(ndim=1, causal=True, dtype="bf16", batch=2, heads=2, n=2048, block=64),
    "map_2d": dict(ndim=2, causal=False, dtype="bf16", batch=1, heads=3, side=48, block=8),
}


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def _draws(name, dev, count=3):
    c = CASES[name]
    out = []
    for i in range(count):
        kw = {"side": c["side"]} if c["ndim"] == 2 else {"n": c["n"]}
        w = fma_inputs.custom("%s_%d" % (name, i), c["ndim"], c["causal"], c["dtype"], c["batch"], c["heads"],
                              block=c["block"], seed=100 + i, **kw)
        out.append(tuple(t.to(dev) for t in fma_inputs.make_inputs(w)))
    return w, out


def _plan(w, linear=False):
    return F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block, causal=w.causal,
                 dtype=w.torch_dtype, side=w.side, linear=linear)


def _load(static, draw):
    for s, d in zip(static, draw):
        s.copy_(d)


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("static_ws", [False, True], ids=["workspace", "static"])
def test_forward_graph_replays(name, static_ws):
    dev = _dev()
    w, draws = _draws(name, dev)
    op = _plan(w)
    ws = op.new_workspace(dev)
    st = [t.clone() for t in draws[0]]
    out = torch.empty_like(st[0])

    def call(buf, o):
        if static_ws:
            return op.forward_static(*buf, out=o)
        return op.forward(*buf, out=o, workspace=ws)

    call(st, out)   # eager first: the launchers' per-device caches are filled outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(st, out)
    ref_ws = op.new_workspace(dev)
    for rep in range(2):
        for i, d in enumerate(draws):
            _load(st, d)
            g.replay()
            ref = op.forward(*d, workspace=ref_ws)   # eager work between the replays
            torch.cuda.synchronize()
            assert torch.equal(out, ref), (name, rep, i)


@pytest.mark.parametrize("name", ["bidi_1d", "map_2d"])
def test_backward_graph_replays(name):
    dev = _dev()
    w, draws = _draws(name, dev)
    op = _plan(w)
    st = [t.clone() for t in draws[0]]
    gen = torch.Generator(device="cpu").manual_seed(7)
    douts = [torch.randn(st[0].shape, generator=gen).to(dev, st[0].dtype) for _ in draws]
    outs = [op.forward(*d) for d in draws]
    o_s, g_s = outs[0].clone(), douts[0].clone()
    bws = torch.empty(max(op.backward_workspace_bytes, 16), dtype=torch.uint8, device=dev)
    op.backward(*st, o_s, g_s, workspace=bws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        grads = op.backward(*st, o_s, g_s, workspace=bws)
    for rep in range(2):
        for i, d in enumerate(draws):
            _load(st, d)
            o_s.copy_(outs[i])
            g_s.copy_(douts[i])
            g.replay()
            ref = op.backward(*d, outs[i], douts[i])
            torch.cuda.synchronize()
            for x, (a, b) in enumerate(zip(grads, ref)):
                assert torch.equal(a, b), (name, rep, i, x)


def test_linear_forward_graph_replays():
    dev = _dev()
    w, draws = _draws("bidi_1d", dev)
    op = _plan(w, linear=True)
    ws = op.new_workspace(dev)
    gen = torch.Generator(device="cpu").manual_seed(11)
    wqs = [torch.rand(d[3].shape, generator=gen).to(dev) for d in draws]
    st = [t.clone() for t in draws[0]]
    wq_s = wqs[0].clone()
    out = torch.empty_like(st[0])
    op.forward_linear(st[0], st[1], st[2], wq_s, st[3], st[4], out=out, workspace=ws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        op.forward_linear(st[0], st[1], st[2], wq_s, st[3], st[4], out=out, workspace=ws)
    ref_ws = op.new_workspace(dev)
    for rep in range(2):
        for i, d in enumerate(draws):
            _load(st, d)
            wq_s.copy_(wqs[i])
            g.replay()
            ref = op.forward_linear(d[0], d[1], d[2], wqs[i], d[3], d[4], workspace=ref_ws)
            torch.cuda.synchronize()
            assert torch.equal(out, ref), (rep, i)
