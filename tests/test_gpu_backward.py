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


def _case(name, ndim, causal, dt, B, H, size, r, p=1, shared=False):
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, causal, dt, B, H, n=size, block=r, seed=seed, rank=p)
    elif isinstance(size, tuple):   # (rows, columns)
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size[1], height=size[0], block=r, seed=seed, rank=p)
    else:
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size, block=r, seed=seed, rank=p)
    q, k, v, wk, wv = fma_inputs.make_inputs(w, weights_shared=shared)
    g = torch.Generator().manual_seed(seed + 1)
    dout = torch.randn(q.shape, generator=g).to(q.dtype)
    return w, q, k, v, wk, wv, dout


def _gpu_backward(w, q, k, v, wk, wv, dout, dev, shared=False, per_level=False):
    op = F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block, causal=w.causal,
               dtype=w.torch_dtype, side=w.side, weights_per_head=not shared, rank=w.rank,
               norm=F.FMA_NORM_PER_LEVEL if per_level else F.FMA_NORM_JOINT)
    t = [x.to(dev) for x in (q, k, v, wk, wv, dout)]
    out = op.forward(*t[:5])
    grads = op.backward(t[0], t[1], t[2], t[3], t[4], out, t[5])
    torch.cuda.synchronize()
    return out.cpu(), [None if x is None else x.cpu() for x in grads]


def _oracle_grads(w, q, k, v, wk, wv, dout, b, h, shared=False, per_level=False):
    pk = None if wk.numel() == 0 else _np(wk if shared else wk[h])
    pv = None if wv.numel() == 0 else _np(wv if shared else wv[h])
    norm = oracle.NORM_PER_SET if per_level else oracle.NORM_JOINT
    if w.ndim == 1:
        return oracle.backward_1d(_np(q[b, h]), _np(k[b, h]), _np(v[b, h]), w.block, pk, pv, _np(dout[b, h]),
                                  causal=w.causal, rank=w.rank, norm=norm)
    return oracle.backward_2d(_np(q[b, h]), _np(k[b, h]), _np(v[b, h]), w.side, w.block, pk, pv,
                              _np(dout[b, h]), rank=w.rank, norm=norm, H=w.rows)


NAMES = ["dq", "dk", "dv", "dwk", "dwv"]


def _check(w, q, k, v, wk, wv, dout, grads, shared=False, per_level=False):
    worst = [[0.0, 0.0] for _ in range(5)]
    refs = {}
    for b in range(w.batch):
        for h in range(w.heads):
            ref = refs[(b, h)] = _oracle_grads(w, q, k, v, wk, wv, dout, b, h, shared, per_level)
            for x in range(3):
                e = parity_record.slice_errors(_np(grads[x][b, h]), ref[x])
                worst[x] = [max(worst[x][0], e[0]), max(worst[x][1], e[1])]
    if grads[3] is not None:
        # weights: the oracle's per-slice gradients summed over the slices that
        # use them (per head: over the batch; shared: over every slice)
        for x in (3, 4):
            if shared:
                acc = sum(refs[bh][x] for bh in refs)
                worst[x] = list(parity_record.slice_errors(_np(grads[x]), acc))
            else:
                for h in range(w.heads):
                    acc = sum(refs[(b, h)][x] for b in range(w.batch))
                    e = parity_record.slice_errors(_np(grads[x][h]), acc)
                    worst[x] = [max(worst[x][0], e[0]), max(worst[x][1], e[1])]
    nrec = 5 if grads[3] is not None else 3
    for x in range(nrec):
        parity_record.record(w.name, NAMES[x], worst[x][0], worst[x][1], TOL[w.dtype],
                             w.batch * w.heads if x < 3 else (1 if shared else w.heads))
    print("%s rel err " % w.name + " ".join("%s %.2e" % (NAMES[x], worst[x][0]) for x in range(nrec)), flush=True)
    for x in range(nrec):
        assert worst[x][0] <= TOL[w.dtype], (w.name, NAMES[x], worst[x][0])


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
    # the printed per-level normalisation: a level's slots padded to 4 (rank
    # 1 in 1D), 8 (rank 2), 16 (rank 3..5), 32 (rank 6..10, 2D)
    ("bwd_pl_bidi_f32_r64", 1, False, "f32", 1, 2, 512, 64, 1, True),
    ("bwd_pl_causal_bf16_r128", 1, True, "bf16", 1, 2, 2048, 128, 1, True),
    ("bwd_pl_p3_bidi_bf16", 1, False, "bf16", 1, 2, 2048, 64, 3, True),
    ("bwd_pl_p10_causal_f32", 1, True, "f32", 1, 1, 1024, 64, 10, True),
    ("bwd_pl_ragged_bf16", 1, False, "bf16", 1, 1, 64 * 11, 64, 1, True),
    ("bwd_pl_r256_p2_bf16", 1, False, "bf16", 1, 2, 2048, 256, 2, True),
    ("bwd_pl_2d_r8_bf16", 2, False, "bf16", 1, 2, 64, 8, 1, True),
    ("bwd_pl_2d_ragged_f32", 2, False, "f32", 1, 1, 40, 8, 1, True),
    ("bwd_pl_2d_r16_bf16", 2, False, "bf16", 1, 1, 64, 16, 1, True),
    # blocks smaller than a wave (1D r = 16, 32; 2D 4 x 4 cells): one chunk
    # per block with idle lanes, near fields packed 64 tokens to a tile
    ("bwd_r16_bidi_bf16", 1, False, "bf16", 1, 2, 1024, 16, 1),
    ("bwd_r16_causal_f32", 1, True, "f32", 1, 2, 512, 16, 1),
    ("bwd_r32_ragged_causal_bf16", 1, True, "bf16", 1, 2, 32 * 23, 32, 1),
    ("bwd_r32_p2_bidi_f32", 1, False, "f32", 1, 1, 1024, 32, 2),
    ("bwd_pl_r16_bf16", 1, False, "bf16", 1, 2, 1024, 16, 1, True),
    ("bwd_2d_r4_bf16", 2, False, "bf16", 1, 2, 32, 4, 1),
    ("bwd_2d_r4_ragged_f32", 2, False, "f32", 1, 1, 44, 4, 1),
    ("bwd_pl_2d_r4_bf16", 2, False, "bf16", 1, 1, 32, 4, 1, True),
    # rectangular maps (rows, columns): wide, tall, ragged on both axes, one
    # row of cells, 16 x 16 and 4 x 4 cells, rank 2, per-level
    ("bwd_rect_wide_bf16", 2, False, "bf16", 1, 2, (32, 64), 8, 1),
    ("bwd_rect_tall_f32", 2, False, "f32", 1, 1, (64, 16), 8, 1),
    ("bwd_rect_ragged_bf16_p2", 2, False, "bf16", 1, 1, (24, 40), 8, 2),
    ("bwd_rect_row_bf16", 2, False, "bf16", 1, 2, (8, 64), 8, 1),
    ("bwd_rect_r16_bf16", 2, False, "bf16", 1, 1, (32, 96), 16, 1),
    ("bwd_rect_r4_f32", 2, False, "f32", 1, 1, (16, 40), 4, 1),
    ("bwd_pl_rect_bf16", 2, False, "bf16", 1, 2, (40, 24), 8, 1, True),
    # 2D per-level at rank p >= 2 (levels of 64 .. 128 slots, whole blocks)
    ("bwd_pl_p2_2d_r8_bf16", 2, False, "bf16", 1, 2, 64, 8, 2, True),
    ("bwd_pl_p3_2d_ragged_f32", 2, False, "f32", 1, 1, 40, 8, 3, True),
    ("bwd_pl_p2_2d_r4_f32", 2, False, "f32", 1, 1, 32, 4, 2, True),
    ("bwd_pl_p4_2d_r16_bf16", 2, False, "bf16", 1, 1, 64, 16, 4, True),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_backward_parity(case):
    dev = _dev()
    per_level = case[9] if len(case) > 9 else False
    w, q, k, v, wk, wv, dout = _case(*case[:9])
    _, grads = _gpu_backward(w, q, k, v, wk, wv, dout, dev, per_level=per_level)
    _check(w, q, k, v, wk, wv, dout, grads, per_level=per_level)


# Score jumps: the query pass takes its reference maximum from a query's
# first block and raises it only when a block's weights would pass 2^64.  On
# peaked inputs (exact integer scores in log2 units) the first channel of
# every fourth key of the second half of the sequence (2D: of the lower half
# of the map) is set to J and every query's first channel to 2, so those
# keys and the coarse rows that aggregate them score about 2J above the
# first block: the raise is taken in near, causal-diagonal and coarse blocks
# (J = 400: past fp32's range without it).  The keys' other channels stay
# distinct, so the softmax over them, and dq, stay far from degenerate.  fp32
# I/O: with a key channel that large in common, dq's sum over the jump keys
# cancels to a small remainder, which bf16 rounding of O (through D = dO . O)
# would swamp -- a conditioning matter, not the raise under test.
BWD_JUMPS = [
    # name, ndim, causal, B, H, n/side, r, J
    ("bwd_jump_bidi_r128", 1, False, 1, 2, 2048, 128, 60),
    ("bwd_jump_causal_r64_overflow", 1, True, 1, 2, 2048, 64, 400),
    ("bwd_jump_2d_r8", 2, False, 1, 2, 64, 8, 400),
]


@pytest.mark.parametrize("case", BWD_JUMPS, ids=[c[0] for c in BWD_JUMPS])
def test_backward_score_jumps(case):
    dev = _dev()
    name, ndim, causal, B, H, size, r, J = case
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, causal, "f32", B, H, n=size, block=r, seed=seed)
    else:
        w = fma_inputs.custom(name, 2, False, "f32", B, H, side=size, block=r, seed=seed)
    q, k, v, wk, wv = fma_inputs.make_peaked_inputs(w)
    idx = torch.arange(w.n // 2, w.n, 4)
    q[..., 0] = 2
    k[:, :, idx, 0] = J
    scale = fma_inputs.PEAKED_SCALE
    dout = torch.randn(q.shape, generator=torch.Generator().manual_seed(seed + 1)).to(q.dtype)
    op = F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block, causal=w.causal,
               dtype=w.torch_dtype, side=w.side, softmax_scale=scale)
    t = [x.to(dev) for x in (q, k, v, wk, wv, dout)]
    out = op.forward(*t[:5])
    grads = [None if x is None else x.cpu() for x in op.backward(t[0], t[1], t[2], t[3], t[4], out, t[5])]
    torch.cuda.synchronize()
    for x in range(3):
        assert torch.isfinite(grads[x].float()).all(), (name, NAMES[x])
    worst = [0.0] * 5
    acc = [0.0, 0.0]
    for b in range(w.batch):
        for h in range(w.heads):
            args = (_np(q[b, h]), _np(k[b, h]), _np(v[b, h]))
            if w.ndim == 1:
                ref = oracle.backward_1d(*args, w.block, _np(wk[h]), _np(wv[h]), _np(dout[b, h]), causal=w.causal,
                                         scale=scale)
            else:
                ref = oracle.backward_2d(*args, w.side, w.block, _np(wk[h]), _np(wv[h]), _np(dout[b, h]),
                                         scale=scale)
            for x in range(3):
                worst[x] = max(worst[x], parity_record.slice_errors(_np(grads[x][b, h]), ref[x])[0])
            for x in (3, 4):
                worst[x] = max(worst[x], parity_record.slice_errors(_np(grads[x][h]), ref[x])[0])
    print("%s rel err " % name + " ".join("%s %.2e" % (NAMES[x], worst[x]) for x in range(5)), flush=True)
    # the jump keys' common channel (J against unit-size channels) scales
    # fp32 rounding in dq's cancelling sum by about J / 4: 1e-3 (without the
    # raise, J = 400 gives non-finite outputs)
    for x in range(5):
        assert worst[x] <= 1e-3, (name, NAMES[x], worst[x])


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


@pytest.mark.parametrize("name,slices,whead", [
    ("C3", [(0, 0), (7, 11)], 11),
    ("C4", [(0, 0), (1, 15)], 15),
    ("C5", [(0, 0), (5, 3), (15, 7)], 7),   # slices 0, 43, 127: three of the six query-pass slice passes
    ("C4_level", [(0, 0), (1, 15)], 15),
    ("C5_level", [(0, 0), (15, 7)], 7),
])
def test_backward_workloads(name, slices, whead):
    """Full-size launch, as the benchmark times it: dq, dk and dv of the
    first and the last (batch, head) slice, and the weight gradients of head
    `whead` (the oracle's per-slice gradients summed over the batch) -- the
    widest sets' reductions (C4: level 8, s = 16384) included."""
    dev = _dev()
    per_level = name.endswith("_level")
    w = fma_inputs.WORKLOADS[name.replace("_level", "")]
    q, k, v, wk, wv = fma_inputs.make_inputs(w)
    g = torch.Generator().manual_seed(7)
    dout = torch.randn(q.shape, generator=g).to(q.dtype)
    _, grads = _gpu_backward(w, q, k, v, wk, wv, dout, dev, per_level=per_level)
    refs = {}

    def ref_of(b, h):
        if (b, h) not in refs:
            refs[(b, h)] = _oracle_grads(w, q, k, v, wk, wv, dout, b, h, per_level=per_level)
        return refs[(b, h)]

    bad = []
    for x in range(3):
        errs = [parity_record.slice_errors(_np(grads[x][b, h]), ref_of(b, h)[x]) for (b, h) in slices]
        worst = max(e[0] for e in errs)
        parity_record.record(name, NAMES[x], worst, max(e[1] for e in errs), TOL[w.dtype], len(slices))
        print(name, NAMES[x], "%.2e" % worst, flush=True)
        if not worst <= TOL[w.dtype]:
            bad.append((NAMES[x], worst))
    for x in (3, 4):
        acc = sum(ref_of(b, whead)[x] for b in range(w.batch))
        e = parity_record.slice_errors(_np(grads[x][whead]), acc)
        parity_record.record(name, NAMES[x], e[0], e[1], TOL[w.dtype], 1)
        print(name, NAMES[x], "head", whead, "%.2e" % e[0], flush=True)
        if not e[0] <= TOL[w.dtype]:
            bad.append((NAMES[x], e[0]))
    assert not bad, (name, bad)
