"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Tolerances: per (batch, head) slice, max|O_gpu - O_ref| / max|O_ref| <= 1e-5
for fp32 and <= 2e-2 for bf16 (the oracle runs in fp64 on the exact bf16
input values).  Index lists are compared bit for bit.  The worst slice's
inf-norm and RMS relative errors of every case are recorded (parity_record)
and printed in the terminal summary.
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
    """max |got - ref| / max |ref| over one slice."""
    return float(np.abs(got - ref).max() / max(np.abs(ref).max(), 1e-30))


def _op(w: fma_inputs.Workload, weights_shared=False, per_level=False):
    return F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block,
                 causal=w.causal, dtype=w.torch_dtype, side=w.side, head_dim=w.head_dim,
                 weights_per_head=not weights_shared, rank=w.rank,
                 norm=F.FMA_NORM_PER_LEVEL if per_level else F.FMA_NORM_JOINT)


def _oracle_slice(w, q, k, v, wk, wv, b, h, weights_shared=False, per_level=False, scale=None):
    pk = None if wk.numel() == 0 else _np(wk if weights_shared else wk[h])
    pv = None if wv.numel() == 0 else _np(wv if weights_shared else wv[h])
    norm = oracle.NORM_PER_SET if per_level else oracle.NORM_JOINT
    if w.ndim == 1:
        return oracle.forward_1d(_np(q[b, h]), _np(k[b, h]), _np(v[b, h]), w.block, pk, pv, causal=w.causal,
                                 rank=w.rank, norm=norm, scale=scale)
    return oracle.forward_2d(_np(q[b, h]), _np(k[b, h]), _np(v[b, h]), w.side, w.block, pk, pv, rank=w.rank,
                             norm=norm, scale=scale, H=w.rows)


def _oracle_all(w, q, k, v, wk, wv, weights_shared=False, per_level=False, scale=None):
    """The oracle on every (batch, head) slice in one call: [B, H, n, d]."""
    pk = None if wk.numel() == 0 else _np(wk)
    pv = None if wv.numel() == 0 else _np(wv)
    norm = oracle.NORM_PER_SET if per_level else oracle.NORM_JOINT
    if w.ndim == 1:
        return oracle.forward_1d(_np(q), _np(k), _np(v), w.block, pk, pv, causal=w.causal, rank=w.rank, norm=norm,
                                 scale=scale)
    return oracle.forward_2d(_np(q), _np(k), _np(v), w.side, w.block, pk, pv, rank=w.rank, norm=norm, scale=scale,
                             H=w.rows)


def _run(w, q, k, v, wk, wv, dev, weights_shared=False, per_level=False, scale=0.0):
    op = F.FMA(ndim=w.ndim, batch=w.batch, heads=w.heads, seq_len=w.n, block=w.block,
               causal=w.causal, dtype=w.torch_dtype, side=w.side, head_dim=w.head_dim,
               weights_per_head=not weights_shared, rank=w.rank, softmax_scale=scale,
               norm=F.FMA_NORM_PER_LEVEL if per_level else F.FMA_NORM_JOINT)
    out = op.forward(q.to(dev), k.to(dev), v.to(dev), wk.to(dev), wv.to(dev))
    torch.cuda.synchronize()
    return op, out.cpu()


def _check_slices(w, q, k, v, wk, wv, out, slices=None, weights_shared=False, per_level=False, scale=None,
                  case=None):
    """Compare the GPU output with the oracle on the given (batch, head)
    slices (None: every slice, one oracle call), hold each slice to the
    dtype's tolerance and record the worst inf-norm and RMS errors."""
    worst = worst_rms = 0.0
    if slices is None:
        ref_all = _oracle_all(w, q, k, v, wk, wv, weights_shared, per_level, scale)
        slices = [(b, h) for b in range(w.batch) for h in range(w.heads)]
    else:
        ref_all = None
    got_all = _np(out)
    bad = []
    for (b, h) in slices:
        ref = ref_all[b, h] if ref_all is not None else _oracle_slice(w, q, k, v, wk, wv, b, h, weights_shared,
                                                                        per_level, scale)
        e, er = parity_record.slice_errors(got_all[b, h], ref)
        worst, worst_rms = max(worst, e), max(worst_rms, er)
        if not e <= TOL[w.dtype]:
            bad.append((b, h, e))
    parity_record.record(case or w.name, "out", worst, worst_rms, TOL[w.dtype], len(slices))
    print("%s worst slice rel err %.3e (rms %.3e) over %d slices" % (case or w.name, worst, worst_rms, len(slices)),
          flush=True)
    assert not bad, (case or w.name, bad[:8])
    return worst


# ------------------------------------------------------------ index lists
@pytest.mark.parametrize("n,r,causal", [(1024, 64, False), (4096, 64, True), (16384, 128, True),
                                        (65536, 128, False), (64 * 11, 64, False), (64 * 13, 64, True),
                                        (128 * 37, 128, False), (192 * 6, 192, True), (16 * 37, 16, True),
                                        (2048, 32, False)])
def test_interaction_lists_1d_bit_exact(n, r, causal):
    dev = _dev()
    op = F.FMA(ndim=1, batch=1, heads=1, seq_len=n, block=r, causal=causal)
    got = op.interaction_lists(dev).cpu().numpy()
    ref, _, _ = oracle.lists_1d(n, r, kcap=3)
    if causal:
        # keep the groups whose tokens are all <= the first row of the block
        L = op.levels
        for b in range(ref.shape[0]):
            for l in range(1, L):
                s = r * 2 ** (l - 1)
                keep = [g for g in ref[b, l - 1] if g >= 0 and min((g + 1) * s, n) - 1 <= b * r]
                ref[b, l - 1] = keep + [-1] * (3 - len(keep))
    assert got.shape == ref.shape
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("W,r", [(128, 8), (64, 16), (40, 8), (256, 8), (96, 16), (64, 4), (44, 4)])
def test_interaction_lists_2d_bit_exact(W, r):
    dev = _dev()
    op = F.FMA(ndim=2, batch=1, heads=1, seq_len=W * W, block=r, side=W)
    got = op.interaction_lists(dev).cpu().numpy()
    ref = oracle.lists_2d(W, r, kcap=27)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("H,W,r", [(32, 64, 8), (128, 32, 8), (24, 40, 8), (8, 64, 8), (64, 8, 8), (96, 160, 8),
                                   (64, 128, 16), (16, 64, 4), (48, 16, 4)])
def test_interaction_lists_2d_rect_bit_exact(H, W, r):
    """Maps of H rows by W columns: the lists against the oracle's set-builder
    lists, bit for bit."""
    dev = _dev()
    op = F.FMA(ndim=2, batch=1, heads=1, seq_len=H * W, block=r, side=W)
    got = op.interaction_lists(dev).cpu().numpy()
    ref = oracle.lists_2d(W, r, kcap=27, H=H)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref)


# ------------------------------------------------------------ coarsening
@pytest.mark.parametrize("name", ["C1", "C2", "small_ragged", "C5s", "2d_ragged", "2d_partial",
                                  "C2_p4", "f32_ragged_p3", "bf16_ragged_p5", "C5s_p4", "2d_f32_p5",
                                  "long_p8", "p4_24sets", "2d_p5_two_passes", "2d_r16_partial", "2d_w32",
                                  "r16_bf16", "r32_f32_p3", "2d_r4_bf16", "2d_r4_f32_ragged", "2d_r4_bf16_p4",
                                  "2d_rect_wide", "2d_rect_tall_partial", "2d_rect_ragged_f32", "2d_rect_r4",
                                  "2d_rect_r16_p2", "2d_rect_row", "d128_1d_bf16", "d32_1d_f32", "d128_2d_r4_f32",
                                  "d32_2d_r8_bf16", "d128_2d_r16_bf16_p2",
                                  "C3", "C4", "C5", "C4_p4", "C5_p4"])
def test_coarsening_parity(name):
    """K_bar, V_bar against the oracle; the rank-p cases cover one pass (at
    most 32 coarse sets in 1D bf16, 32 accumulator columns in 2D bf16, 16
    sets in fp32) and several (up to 64 sets)."""
    dev = _dev()
    ws = {
        "C1": fma_inputs.WORKLOADS["C1"],
        "C2": fma_inputs.WORKLOADS["C2"],
        "small_ragged": fma_inputs.custom("small_ragged", 1, False, "bf16", 2, 3, 64 * 23, block=64, seed=5),
        "C5s": fma_inputs.custom("C5s", 2, False, "bf16", 1, 2, side=128, block=8, seed=6),
        "2d_ragged": fma_inputs.custom("2d_ragged", 2, False, "f32", 1, 2, side=8 * 11, block=8, seed=7),
        "2d_partial": fma_inputs.custom("2d_partial", 2, False, "bf16", 1, 1, side=256, block=8, seed=8),
        "C2_p4": fma_inputs.with_rank(fma_inputs.WORKLOADS["C2"], 4),
        "f32_ragged_p3": fma_inputs.custom("f32_ragged_p3", 1, False, "f32", 1, 2, 64 * 23, block=64, seed=9,
                                           rank=3),
        "bf16_ragged_p5": fma_inputs.custom("bf16_ragged_p5", 1, False, "bf16", 1, 2, 128 * 37, block=128,
                                            seed=10, rank=5),
        "C5s_p4": fma_inputs.custom("C5s_p4", 2, False, "bf16", 1, 2, side=128, block=8, seed=11, rank=4),
        "2d_f32_p5": fma_inputs.custom("2d_f32_p5", 2, False, "f32", 1, 1, side=8 * 11, block=8, seed=12,
                                       rank=5),
        "long_p8": fma_inputs.custom("long_p8", 1, False, "bf16", 1, 1, 65536, block=128, seed=13, rank=8),
        # 24 sets in one 1D pass; 2D: 35 columns (two passes), 64-pixel
        # squares wider than a tile (partials), the smallest map with a level
        "p4_24sets": fma_inputs.custom("p4_24sets", 1, False, "bf16", 1, 2, 16384, block=128, seed=14, rank=4),
        "2d_p5_two_passes": fma_inputs.custom("2d_p5_two_passes", 2, False, "bf16", 1, 2, side=128, block=8,
                                              seed=15, rank=5),
        "2d_r16_partial": fma_inputs.custom("2d_r16_partial", 2, False, "bf16", 1, 2, side=128, block=16, seed=16,
                                            rank=2),
        "2d_w32": fma_inputs.custom("2d_w32", 2, False, "bf16", 2, 2, side=32, block=8, seed=17),
        # small blocks: the chunk kernel for 1D bf16, 64-run tiles for 4 x 4 cells
        "r16_bf16": fma_inputs.custom("r16_bf16", 1, False, "bf16", 2, 2, 4096, block=16, seed=18),
        "r32_f32_p3": fma_inputs.custom("r32_f32_p3", 1, False, "f32", 1, 2, 32 * 45, block=32, seed=19, rank=3),
        "2d_r4_bf16": fma_inputs.custom("2d_r4_bf16", 2, False, "bf16", 1, 2, side=128, block=4, seed=20),
        "2d_r4_f32_ragged": fma_inputs.custom("2d_r4_f32_ragged", 2, False, "f32", 1, 2, side=4 * 11, block=4,
                                              seed=21),
        "2d_r4_bf16_p4": fma_inputs.custom("2d_r4_bf16_p4", 2, False, "bf16", 1, 1, side=64, block=4, seed=22,
                                           rank=4),
        # rectangular maps (H rows by W columns): whole 32x32 tiles (streaming
        # kernel), squares wider than a tile along both axes, ragged axes
        # (tile kernel), 4 x 4 cells, rank 2, a single row of cells
        "2d_rect_wide": fma_inputs.custom("2d_rect_wide", 2, False, "bf16", 2, 2, side=64, height=32, block=8,
                                          seed=23),
        "2d_rect_tall_partial": fma_inputs.custom("2d_rect_tall_partial", 2, False, "bf16", 1, 2, side=64,
                                                  height=256, block=8, seed=24),
        "2d_rect_ragged_f32": fma_inputs.custom("2d_rect_ragged_f32", 2, False, "f32", 1, 2, side=40, height=24,
                                                block=8, seed=25),
        "2d_rect_r4": fma_inputs.custom("2d_rect_r4", 2, False, "bf16", 1, 2, side=128, height=16, block=4,
                                        seed=26),
        "2d_rect_r16_p2": fma_inputs.custom("2d_rect_r16_p2", 2, False, "bf16", 1, 2, side=128, height=64,
                                            block=16, seed=27, rank=2),
        "2d_rect_row": fma_inputs.custom("2d_rect_row", 2, False, "bf16", 1, 1, side=96, height=8, block=8,
                                         seed=28),
        # head dims 32 and 128 (chunk and tile kernels; 4 x 4 cells at d = 128
        # take 1024-thread tiles)
        "d128_1d_bf16": fma_inputs.custom("d128_1d_bf16", 1, False, "bf16", 2, 2, 64 * 23, block=64, seed=29,
                                          head_dim=128),
        "d32_1d_f32": fma_inputs.custom("d32_1d_f32", 1, False, "f32", 1, 2, 4096, block=128, seed=30, head_dim=32),
        "d128_2d_r4_f32": fma_inputs.custom("d128_2d_r4_f32", 2, False, "f32", 1, 2, side=44, block=4, seed=31,
                                            head_dim=128),
        "d32_2d_r8_bf16": fma_inputs.custom("d32_2d_r8_bf16", 2, False, "bf16", 1, 2, side=128, block=8, seed=32,
                                            head_dim=32),
        "d128_2d_r16_bf16_p2": fma_inputs.custom("d128_2d_r16_bf16_p2", 2, False, "bf16", 1, 2, side=128,
                                                 block=16, seed=33, rank=2, head_dim=128),
    }
    for full in ("C3", "C4", "C5"):   # the bench's workloads at full size, every slice
        ws[full] = fma_inputs.WORKLOADS[full]
        ws[full + "_p4"] = fma_inputs.with_rank(fma_inputs.WORKLOADS[full], 4)
    w = ws[name]
    q, k, v, wk, wv = fma_inputs.make_inputs(w)
    op = _op(w)
    work = op.coarsen(k.to(dev), v.to(dev), wk.to(dev), wv.to(dev))
    torch.cuda.synchronize()
    kb, vb = [t.cpu() for t in op.coarse_views(work)]
    worst = {"K_bar": [0.0, 0.0], "V_bar": [0.0, 0.0]}
    count = 0
    for b in range(w.batch):
        for h in range(w.heads):
            if w.ndim == 1:
                rk = oracle.coarsen_1d(_np(k[b, h]), w.block, _np(wk[h]), rank=w.rank)
                rv = oracle.coarsen_1d(_np(v[b, h]), w.block, _np(wv[h]), rank=w.rank)
            else:
                rk = oracle.coarsen_2d(_np(k[b, h]), w.side, w.block, _np(wk[h]), rank=w.rank, H=w.rows)
                rv = oracle.coarsen_2d(_np(v[b, h]), w.side, w.block, _np(wv[h]), rank=w.rank, H=w.rows)
            for t, got, ref in (("K_bar", kb[b, h], rk), ("V_bar", vb[b, h], rv)):
                e, er = parity_record.slice_errors(_np(got), ref)
                worst[t] = [max(worst[t][0], e), max(worst[t][1], er)]
                assert e <= TOL[w.dtype], (name, t, b, h, e)
            count += 1
    for t, (e, er) in worst.items():
        parity_record.record("coarsen_" + name, t, e, er, TOL[w.dtype], count)


# ------------------------------------------------------------ forward, small
SMALL = [
    # name, ndim, causal, dtype, B, H, n/side, block
    ("bidi_f32_r64", 1, False, "f32", 1, 2, 1024, 64),
    ("causal_f32_r64", 1, True, "f32", 1, 2, 1024, 64),
    ("bidi_bf16_r128", 1, False, "bf16", 2, 2, 4096, 128),
    ("causal_bf16_r128", 1, True, "bf16", 2, 2, 4096, 128),
    ("ragged_bidi_bf16", 1, False, "bf16", 1, 3, 64 * 23, 64),
    ("ragged_causal_bf16", 1, True, "bf16", 1, 3, 64 * 21, 64),
    ("ragged_causal_f32", 1, True, "f32", 1, 1, 128 * 11, 128),
    ("r192_bidi_bf16", 1, False, "bf16", 1, 2, 192 * 10, 192),
    ("r256_causal_bf16", 1, True, "bf16", 1, 2, 256 * 8, 256),
    ("single_block", 1, False, "bf16", 1, 2, 64, 64),
    ("two_blocks_causal", 1, True, "f32", 1, 2, 128, 64),
    ("2d_r8_bf16", 2, False, "bf16", 2, 2, 64, 8),
    ("2d_r8_f32", 2, False, "f32", 1, 2, 32, 8),
    ("2d_r16_bf16", 2, False, "bf16", 1, 2, 64, 16),
    ("2d_ragged_bf16", 2, False, "bf16", 1, 2, 40, 8),
    ("2d_ragged_r16_f32", 2, False, "f32", 1, 1, 80, 16),
    ("2d_single_cell", 2, False, "bf16", 1, 1, 8, 8),
    # coarse level rank p (p basis vectors per level): one coarsening pass
    # and several, up to the 64-set limit
    ("p4_bidi_bf16_r64", 1, False, "bf16", 1, 2, 2048, 64, 4),
    ("p4_causal_bf16_r128", 1, True, "bf16", 1, 2, 16384, 128, 4),
    ("p3_causal_f32_r64", 1, True, "f32", 1, 2, 1024, 64, 3),
    ("p5_ragged_bidi_f32", 1, False, "f32", 1, 1, 64 * 23, 64, 5),
    ("p2_ragged_causal_bf16", 1, True, "bf16", 1, 2, 64 * 21, 64, 2),
    ("p8_bidi_bf16_64sets", 1, False, "bf16", 1, 1, 65536, 128, 8),
    ("p4_2d_r8_bf16", 2, False, "bf16", 1, 2, 64, 8, 4),
    ("p5_2d_r8_bf16_15sets", 2, False, "bf16", 1, 1, 128, 8, 5),
    ("p5_2d_ragged_f32", 2, False, "f32", 1, 1, 40, 8, 5),
    ("p3_2d_r16_bf16", 2, False, "bf16", 1, 1, 64, 16, 3),
    # the printed per-level normalisation (level slots padded to 4, 8, 16, 32)
    ("pl_bidi_f32_r64", 1, False, "f32", 1, 2, 1024, 64, 1, True),
    ("pl_causal_bf16_r128", 1, True, "bf16", 2, 2, 4096, 128, 1, True),
    ("pl_ragged_causal_bf16", 1, True, "bf16", 1, 3, 64 * 21, 64, 1, True),
    ("pl_ragged_bidi_f32", 1, False, "f32", 1, 1, 128 * 11, 128, 1, True),
    ("pl_p2_bidi_bf16", 1, False, "bf16", 1, 2, 2048, 64, 2, True),
    ("pl_p3_causal_f32", 1, True, "f32", 1, 2, 1024, 64, 3, True),
    ("pl_p4_causal_bf16_r128", 1, True, "bf16", 1, 2, 16384, 128, 4, True),
    ("pl_p10_bidi_bf16", 1, False, "bf16", 1, 1, 2048, 64, 10, True),
    ("pl_r256_bidi_bf16", 1, False, "bf16", 1, 2, 256 * 8, 256, 1, True),
    ("pl_2d_r8_bf16", 2, False, "bf16", 2, 2, 64, 8, 1, True),
    ("pl_2d_ragged_f32", 2, False, "f32", 1, 1, 40, 8, 1, True),
    ("pl_2d_r16_bf16", 2, False, "bf16", 1, 2, 64, 16, 1, True),
    # blocks smaller than a wave (1D r = 16, 32; 2D 4 x 4 cells, Sec. 4's
    # block-size sweep): one wave per block, near tiles packed 64 tokens
    # to a tile with the rest masked
    ("r16_bidi_bf16", 1, False, "bf16", 2, 2, 1024, 16),
    ("r16_causal_f32", 1, True, "f32", 1, 2, 1024, 16),
    ("r16_ragged_causal_bf16", 1, True, "bf16", 1, 3, 16 * 37, 16),
    ("r32_bidi_f32", 1, False, "f32", 1, 2, 2048, 32),
    ("r32_ragged_bidi_bf16", 1, False, "bf16", 1, 2, 32 * 23, 32),
    ("r32_causal_bf16_p2", 1, True, "bf16", 1, 2, 4096, 32, 2),
    ("r16_single_block", 1, False, "bf16", 1, 2, 16, 16),
    ("pl_r16_causal_bf16", 1, True, "bf16", 1, 2, 2048, 16, 1, True),
    ("pl_r32_bidi_f32_p3", 1, False, "f32", 1, 1, 1024, 32, 3, True),
    ("2d_r4_bf16", 2, False, "bf16", 2, 2, 64, 4),
    ("2d_r4_f32", 2, False, "f32", 1, 2, 32, 4),
    ("2d_r4_ragged_bf16", 2, False, "bf16", 1, 2, 44, 4),
    ("2d_r4_single_cell", 2, False, "bf16", 1, 1, 4, 4),
    ("p3_2d_r4_bf16", 2, False, "bf16", 1, 1, 32, 4, 3),
    ("pl_2d_r4_bf16", 2, False, "bf16", 1, 2, 64, 4, 1, True),
    ("pl_2d_r4_ragged_f32", 2, False, "f32", 1, 1, 44, 4, 1, True),
    # rectangular maps, (rows, columns): wide and tall (cells in pairs along
    # a row when the cell columns are even), ragged on both axes, odd cell
    # columns, one row or one column of cells, 16 x 16 and 4 x 4 cells, rank
    # and per-level normalisation
    ("rect_wide_bf16", 2, False, "bf16", 2, 2, (32, 64), 8),
    ("rect_tall_bf16", 2, False, "bf16", 1, 2, (128, 32), 8),
    ("rect_ragged_f32", 2, False, "f32", 1, 2, (24, 40), 8),
    ("rect_odd_cols_bf16", 2, False, "bf16", 1, 2, (40, 24), 8),
    ("rect_row_bf16", 2, False, "bf16", 1, 2, (8, 64), 8),
    ("rect_column_f32", 2, False, "f32", 1, 1, (64, 8), 8),
    ("rect_r16_bf16", 2, False, "bf16", 1, 2, (64, 128), 16),
    ("rect_r4_bf16", 2, False, "bf16", 1, 2, (16, 64), 4),
    ("rect_r4_f32", 2, False, "f32", 1, 1, (48, 16), 4),
    ("p3_rect_bf16", 2, False, "bf16", 1, 1, (96, 64), 8, 3),
    ("pl_rect_bf16", 2, False, "bf16", 1, 2, (32, 64), 8, 1, True),
    ("pl_rect_r4_f32", 2, False, "f32", 1, 1, (16, 40), 4, 1, True),
    ("rect_large_bf16", 2, False, "bf16", 2, 2, (96, 160), 8),
    # 2D per-level normalisation at rank p >= 2: a level's 27p slots fill
    # whole 32-slot blocks (64, 96, 128, 160), normalised online over them --
    # within one tile, across tiles, on the fused bf16 kernel (8 x 8 and
    # 16 x 16 cells) and the register-staged one (fp32, 4 x 4 cells)
    ("pl_p2_2d_r8_bf16", 2, False, "bf16", 1, 2, 64, 8, 2, True),
    ("pl_p3_2d_ragged_f32", 2, False, "f32", 1, 1, 40, 8, 3, True),
    ("pl_p4_2d_r16_bf16", 2, False, "bf16", 1, 2, 64, 16, 4, True),
    ("pl_p2_2d_r4_bf16", 2, False, "bf16", 1, 1, 32, 4, 2, True),
    ("pl_p5_2d_r8_bf16", 2, False, "bf16", 1, 1, 64, 8, 5, True),
    ("pl_p3_2d_r8_bf16_3lev", 2, False, "bf16", 1, 2, 128, 8, 3, True),
    ("pl_p2_rect_bf16", 2, False, "bf16", 1, 2, (32, 64), 8, 2, True),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_forward_parity_small(case):
    dev = _dev()
    name, ndim, causal, dt, B, H, size, r = case[:8]
    p = case[8] if len(case) > 8 else 1
    per_level = case[9] if len(case) > 9 else False
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, causal, dt, B, H, n=size, block=r, seed=seed, rank=p)
    elif isinstance(size, tuple):
        w = fma_inputs.custom(name, 2, causal, dt, B, H, side=size[1], height=size[0], block=r, seed=seed, rank=p)
    else:
        w = fma_inputs.custom(name, 2, causal, dt, B, H, side=size, block=r, seed=seed, rank=p)
    q, k, v, wk, wv = fma_inputs.make_inputs(w)
    _, out = _run(w, q, k, v, wk, wv, dev, per_level=per_level)
    _check_slices(w, q, k, v, wk, wv, out, per_level=per_level)


# head dims 32 and 128 (the register-staged kernel and the chunk / tile
# coarsening; d = 64 keeps the matrix-core kernels): 1D bidirectional and
# causal, ragged, blocks of 16 to 256, 2D cells of 4 to 16, rectangular,
# rank p, per-level (also levels of several blocks), fp32 and bf16
HEADDIM = [
    # name, ndim, causal, dtype, B, H, n / side or (rows, cols), block, rank, per_level, d
    ("d32_bidi_bf16_r64", 1, False, "bf16", 2, 2, 1024, 64, 1, False, 32),
    ("d128_causal_bf16_r128", 1, True, "bf16", 1, 2, 4096, 128, 1, False, 128),
    ("d128_bidi_f32_r64", 1, False, "f32", 1, 2, 1024, 64, 1, False, 128),
    ("d32_causal_f32_r16", 1, True, "f32", 1, 2, 16 * 37, 16, 1, False, 32),
    ("d128_ragged_bidi_bf16", 1, False, "bf16", 1, 3, 64 * 23, 64, 1, False, 128),
    ("d128_r256_causal_bf16", 1, True, "bf16", 1, 1, 256 * 8, 256, 1, False, 128),
    ("d32_r32_bidi_bf16_p3", 1, False, "bf16", 1, 2, 32 * 45, 32, 3, False, 32),
    ("d128_p4_bidi_bf16", 1, False, "bf16", 1, 2, 4096, 64, 4, False, 128),
    ("d32_pl_causal_bf16", 1, True, "bf16", 1, 2, 2048, 64, 2, True, 32),
    ("d128_2d_r8_bf16", 2, False, "bf16", 1, 2, 64, 8, 1, False, 128),
    ("d32_2d_r4_bf16", 2, False, "bf16", 1, 2, 32, 4, 1, False, 32),
    ("d128_2d_r4_f32", 2, False, "f32", 1, 1, 44, 4, 1, False, 128),
    ("d128_2d_r16_bf16", 2, False, "bf16", 1, 2, 64, 16, 1, False, 128),
    ("d128_pl_2d_p2_bf16", 2, False, "bf16", 1, 2, 64, 8, 2, True, 128),
    ("d32_rect_f32", 2, False, "f32", 1, 2, (24, 40), 8, 1, False, 32),
    ("d128_rect_bf16_p2", 2, False, "bf16", 1, 2, (32, 64), 8, 2, False, 128),
]


@pytest.mark.parametrize("case", HEADDIM, ids=[c[0] for c in HEADDIM])
def test_forward_parity_head_dims(case):
    dev = _dev()
    name, ndim, causal, dt, B, H, size, r, p, per_level, d = case
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, causal, dt, B, H, n=size, block=r, seed=seed, rank=p, head_dim=d)
    elif isinstance(size, tuple):
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size[1], height=size[0], block=r, seed=seed, rank=p,
                              head_dim=d)
    else:
        w = fma_inputs.custom(name, 2, False, dt, B, H, side=size, block=r, seed=seed, rank=p, head_dim=d)
    q, k, v, wk, wv = fma_inputs.make_inputs(w)
    assert q.shape[-1] == d
    _, out = _run(w, q, k, v, wk, wv, dev, per_level=per_level)
    _check_slices(w, q, k, v, wk, wv, out, per_level=per_level)


def test_forward_shared_weights():
    dev = _dev()
    w = fma_inputs.custom("shared", 1, True, "bf16", 2, 3, n=2048, block=64, seed=11)
    q, k, v, wk, wv = fma_inputs.make_inputs(w, weights_shared=True)
    _, out = _run(w, q, k, v, wk, wv, dev, weights_shared=True)
    _check_slices(w, q, k, v, wk, wv, out, [(0, 0), (1, 2)], weights_shared=True)


def test_empty_batch_is_noop():
    dev = _dev()
    op = F.FMA(ndim=1, batch=0, heads=4, seq_len=1024, block=64)
    x = torch.empty((0, 4, 1024, 64), dtype=torch.bfloat16, device=dev)
    wk = torch.zeros((4, op.weights_len), device=dev)
    out = op.forward(x, x, x, wk, wk, workspace=torch.empty(16, dtype=torch.uint8, device=dev))
    torch.cuda.synchronize()
    assert out.shape == x.shape


# ------------------------------------------------------------ invariants
def test_weights_sum_to_one_gpu():
    """V = 1 and pi^v_l = 1/s_l (every basis) give O = 1 (the joint softmax is
    a convex combination)."""
    dev = _dev()
    for dt, tol, p in (("f32", 1e-6, 1), ("bf16", 1e-2, 1), ("bf16", 1e-2, 3)):
        w = fma_inputs.custom("ones", 1, False, dt, 1, 2, n=4096, block=64, seed=3, rank=p)
        q, k, _, wk, wv = fma_inputs.make_inputs(w)
        v = torch.ones_like(q)
        L = oracle.num_levels(w.n // w.block)
        wv = torch.cat([torch.full((2, 64 * 2 ** (l - 1)), 1.0 / (64 * 2 ** (l - 1)))
                        for l in range(1, L) for _ in range(p)], 1)
        _, out = _run(w, q, k, v, wk, wv, dev)
        assert (out.float() - 1).abs().max().item() <= tol


def test_per_level_weights_sum_to_one_per_set_gpu():
    """Printed form with V = 1 and pi^v_l = 1/s_l: each non-empty set adds 1,
    so a row holds 1 + (its number of non-empty levels) (oracle on the same
    inputs for the count)."""
    dev = _dev()
    for dt, tol, p, causal in (("f32", 1e-5, 1, False), ("bf16", 2e-2, 1, True), ("bf16", 2e-2, 4, False)):
        w = fma_inputs.custom("ones_pl", 1, causal, dt, 1, 1, n=2048, block=64, seed=4, rank=p)
        q, k, _, wk, wv = fma_inputs.make_inputs(w)
        v = torch.ones_like(q)
        L = oracle.num_levels(w.n // w.block)
        wv = torch.cat([torch.full((1, 64 * 2 ** (l - 1)), 1.0 / (64 * 2 ** (l - 1)))
                        for l in range(1, L) for _ in range(p)], 1)
        _, out = _run(w, q, k, v, wk, wv, dev, per_level=True)
        ref = _oracle_slice(w, q, k, v, wk, wv, 0, 0, per_level=True)
        assert ref.max() > 2.5   # rows see several levels
        assert np.abs(_np(out[0, 0]) - ref).max() / ref.max() <= tol


@pytest.mark.parametrize("p", [1, 4])
def test_causality_bit_exact_gpu(p):
    dev = _dev()
    w = fma_inputs.custom("causal", 1, True, "bf16", 1, 2, n=4096, block=64, seed=21, rank=p)
    q, k, v, wk, wv = fma_inputs.make_inputs(w)
    op = _op(w)
    base = op.forward(q.to(dev), k.to(dev), v.to(dev), wk.to(dev), wv.to(dev)).cpu()
    g = torch.Generator().manual_seed(5)
    for t in (63, 64, 1000, 4000):
        q2, k2, v2 = q.clone(), k.clone(), v.clone()
        for a in (q2, k2, v2):
            a[:, :, t + 1:] = (torch.randn(a[:, :, t + 1:].shape, generator=g) * 3).to(a.dtype)
        out = op.forward(q2.to(dev), k2.to(dev), v2.to(dev), wk.to(dev), wv.to(dev)).cpu()
        assert torch.equal(out[:, :, :t + 1], base[:, :, :t + 1])


def test_deterministic_gpu():
    dev = _dev()
    w = fma_inputs.custom("det", 1, False, "bf16", 2, 4, n=8192, block=128, seed=31)
    q, k, v, wk, wv = [t.to(dev) for t in fma_inputs.make_inputs(w)]
    op = _op(w)
    a = op.forward(q, k, v, wk, wv)
    b = op.forward(q, k, v, wk, wv)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# ------------------------------------------------------------ the five workloads
@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5", "C3_p4", "C4_p4", "C5_p4", "C3_level", "C4_level",
                                  "C5_level", "C4_p4_level", "C5_p4_level"])
def test_forward_parity_workloads(name):
    """Full-size launch (as the benchmark times it), every (batch, head)
    slice against the oracle; _p4: the same workload with rank 4 (the paper's
    experimental setting); _level: the printed per-level normalisation."""
    dev = _dev()
    per_level = name.endswith("_level")
    base, _, p = name.replace("_level", "").partition("_p")
    w = fma_inputs.WORKLOADS[base]
    if p:
        w = fma_inputs.with_rank(w, int(p))
    q, k, v, wk, wv = fma_inputs.make_inputs(w)
    _, out = _run(w, q, k, v, wk, wv, dev, per_level=per_level)
    assert torch.isfinite(out.float()).all()
    _check_slices(w, q, k, v, wk, wv, out, per_level=per_level, case=name)


# ------------------------------------------------------------ score jumps
# The fused kernel takes its reference maximum from a query's first block and
# raises it only when a half-block's weights would pass 2^64 (a score more
# than ~60 above it in log2 units).  On peaked inputs (exact integer scores
# in log2 units, fma_inputs.make_peaked_inputs) every fourth key of the
# second half of the sequence (2D: of the lower half of the map) is set to
# (J, 0, ..., 0) and every query's first channel to 2: those keys, and the
# coarse rows that aggregate them, score 2J, up to 2J - 16 above the first
# block's maximum -- past fp32's range without the raise for J = 400 -- in
# near, causal-diagonal, coarse and per-level blocks; J = 20 stays below it.
JUMPS = [
    # name, ndim, causal, B, H, n/side, r, rank, per_level, J
    ("jump_bidi_r128", 1, False, 1, 2, 4096, 128, 1, False, 60),
    ("jump_bidi_r128_overflow", 1, False, 1, 2, 4096, 128, 1, False, 400),
    ("jump_causal_r64", 1, True, 1, 2, 2048, 64, 1, False, 60),
    ("jump_bidi_r128_mild", 1, False, 1, 2, 4096, 128, 1, False, 20),
    ("jump_2d_pairs", 2, False, 1, 2, 64, 8, 1, False, 400),
    ("jump_2d_r16", 2, False, 1, 2, 64, 16, 1, False, 60),
    ("jump_level_causal", 1, True, 1, 2, 4096, 128, 1, True, 60),
    ("jump_2d_level_p2", 2, False, 1, 2, 64, 8, 2, True, 400),
    ("jump_p4_bidi", 1, False, 1, 2, 4096, 64, 4, False, 60),
]


@pytest.mark.parametrize("case", JUMPS, ids=[c[0] for c in JUMPS])
def test_score_jumps(case):
    dev = _dev()
    name, ndim, causal, B, H, size, r, p, per_level, J = case
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, causal, "bf16", B, H, n=size, block=r, seed=seed, rank=p)
    else:
        w = fma_inputs.custom(name, 2, False, "bf16", B, H, side=size, block=r, seed=seed, rank=p)
    q, k, v, wk, wv = fma_inputs.make_peaked_inputs(w)
    idx = torch.arange(w.n // 2, w.n, 4)
    q[..., 0] = 2
    k[:, :, idx, :] = 0
    k[:, :, idx, 0] = J
    scale = fma_inputs.PEAKED_SCALE
    _, out = _run(w, q, k, v, wk, wv, dev, per_level=per_level, scale=scale)
    assert torch.isfinite(out.float()).all(), name
    _check_slices(w, q, k, v, wk, wv, out, per_level=per_level, scale=scale, case=name)


# ------------------------------------------------------------ peaked structure
# Integer queries and keys, one-hot aggregation weights and a softmax scale
# that makes the base-2 scores exact integer dot products
# (fma_inputs.make_peaked_inputs): every row's softmax is dominated by one or
# two sources, so a dropped, duplicated or wrongly masked source -- a far
# group of any level, a slot next to the padding, the causal diagonal --
# moves its rows by about the size of a value vector rather than by a few per
# cent (tests/test_structural_pins.py shows this on the CPU).  The bf16 hot
# kernel computes these scores exactly; only P and the output are rounded.
PEAKED = [
    # name, ndim, causal, B, H, n/side, r, rank, per_level
    ("peaked_C4", 1, False, 2, 16, 65536, 128, 1, False),
    ("peaked_C3", 1, True, 8, 12, 16384, 128, 1, False),
    ("peaked_C5", 2, False, 16, 8, 128, 8, 1, False),
    ("peaked_causal_r64_ragged", 1, True, 1, 4, 64 * 45, 64, 1, False),
    ("peaked_bidi_r256", 1, False, 1, 4, 256 * 16, 256, 1, False),
    ("peaked_causal_r192", 1, True, 1, 2, 192 * 12, 192, 1, False),
    ("peaked_p4_bidi", 1, False, 1, 4, 16384, 128, 4, False),
    ("peaked_p4_causal", 1, True, 1, 4, 8192, 64, 4, False),
    ("peaked_level_causal", 1, True, 1, 4, 8192, 128, 1, True),
    ("peaked_2d_r16", 2, False, 1, 4, 128, 16, 1, False),
    ("peaked_2d_ragged", 2, False, 1, 4, 8 * 13, 8, 1, False),
    ("peaked_2d_p4", 2, False, 1, 2, 64, 8, 4, False),
    ("peaked_2d_level", 2, False, 1, 4, 128, 8, 1, True),
    ("peaked_causal_r16", 1, True, 1, 4, 16 * 45, 16, 1, False),
    ("peaked_bidi_r32_p2", 1, False, 1, 2, 4096, 32, 2, False),
    ("peaked_2d_r4", 2, False, 1, 4, 44, 4, 1, False),
    ("peaked_2d_p2_level", 2, False, 1, 4, 128, 8, 2, True),
]


@pytest.mark.parametrize("case", PEAKED, ids=[c[0] for c in PEAKED])
def test_peaked_structure(case):
    dev = _dev()
    name, ndim, causal, B, H, size, r, p, per_level = case
    seed = zlib.crc32(name.encode()) % 1000
    if ndim == 1:
        w = fma_inputs.custom(name, 1, causal, "bf16", B, H, n=size, block=r, seed=seed, rank=p)
    else:
        w = fma_inputs.custom(name, 2, False, "bf16", B, H, side=size, block=r, seed=seed, rank=p)
    q, k, v, wk, wv = fma_inputs.make_peaked_inputs(w)
    scale = fma_inputs.PEAKED_SCALE
    _, out = _run(w, q, k, v, wk, wv, dev, per_level=per_level, scale=scale)
    _check_slices(w, q, k, v, wk, wv, out, per_level=per_level, scale=scale, case=name)


def test_dense_reference_matches_sdpa():
    dev = _dev()
    for causal in (False, True):
        w = fma_inputs.custom("dense", 1, causal, "bf16", 1, 2, n=2048, block=64, seed=41)
        q, k, v, _, _ = fma_inputs.make_inputs(w)
        op = _op(w)
        out = op.dense_reference(q.to(dev), k.to(dev), v.to(dev)).cpu()
        ref = torch.nn.functional.scaled_dot_product_attention(q.double(), k.double(), v.double(),
                                                               is_causal=causal)
        for h in range(2):
            assert rel_err(_np(out[0, h]), ref[0, h].numpy()) <= 2e-2
