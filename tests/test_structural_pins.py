"""Sensitivity of the peaked-input parity check (CPU, test infrastructure).

The GPU structural test (tests/test_gpu_parity.py::test_peaked_structure_*)
compares the bf16 hot kernel with the oracle on inputs from
fma_inputs.make_peaked_inputs: integer queries and keys, one-hot aggregation
weights and a softmax scale that makes the base-2 scores plain integer dot
products.  Those inputs make every row's softmax sharply peaked, so a source
that is dropped, added or masked wrongly moves some rows by about the size of
a value vector instead of a few per cent.

These tests show that on the CPU, with the mistakes planted in an
independent dense formulation (the n x (n + R) masked score matrix of
oracle/brute.py): each plausible structural mistake -- a whole level dropped,
one list entry per level dropped, a near block dropped, a future token or a
non-past group leaked into a causal row, an empty list slot read as coarse
row 0, a weight offset off by one -- moves the output by far more than the
2e-2 bf16 tolerance, while the unperturbed formulation matches the oracle to
fp64 rounding.
"""
import numpy as np
import pytest
import torch

import fma_inputs
import oracle
from oracle import brute

TOL_BF16 = 2e-2
MIN_MOVE = 0.25   # a planted mistake must move the slice by at least this (relative, inf-norm)


def _rel(a, b):
    return float(np.abs(a - b).max() / np.abs(b).max())


def _inputs(ndim, causal, size, r, seed):
    if ndim == 1:
        w = fma_inputs.custom("peaked", 1, causal, "bf16", 1, 1, n=size, block=r, seed=seed)
    else:
        w = fma_inputs.custom("peaked", 2, False, "bf16", 1, 1, side=size, block=r, seed=seed)
    q, k, v, wk, wv = fma_inputs.make_peaked_inputs(w)
    f = lambda t: t[0, 0].double().numpy()   # noqa: E731
    return w, f(q), f(k), f(v), wk[0].double().numpy(), wv[0].double().numpy()


def _augmented_1d(n, r, k, v, pk, pv):
    kaug = np.vstack([k, brute.aggregation_matrix_1d(n, r, pk) @ k])
    vaug = np.vstack([v, brute.aggregation_matrix_1d(n, r, pv) @ v])
    return kaug, vaug


def _level_offsets_1d(n, r):
    L = oracle.num_levels(n // r)
    sizes = [r * 2 ** (l - 1) for l in range(1, L)]
    counts = [-(-n // s) for s in sizes]
    return sizes, np.cumsum([0] + counts)


@pytest.mark.parametrize("causal", [False, True])
def test_peaked_inputs_are_exact_and_peaked_1d(causal):
    n, r = 512, 32
    w, q, k, v, pk, pv = _inputs(1, causal, n, r, 11 + causal)
    scale = fma_inputs.PEAKED_SCALE
    out = oracle.forward_1d(q, k, v, r, pk, pv, causal=causal, scale=scale)
    kaug, vaug = _augmented_1d(n, r, k, v, pk, pv)
    mask = brute.mask_1d(n, r, causal)
    ref = brute.masked_attention(q, kaug, vaug, mask, scale)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    # every coarse key is one token of its group, bit for bit
    assert set(np.unique(kaug[n:])) <= set(np.unique(k))
    # scores in base-2 units are integers: scale * log2(e) == 1 in float32
    assert np.float32(scale) * np.float32(1.4426950408889634) == np.float32(1.0)
    s = q @ kaug.T
    assert np.array_equal(s, np.round(s))
    # peaked: the top source carries a large share of the weight in most rows
    # (integer scores tie now and then, which splits the top weight)
    z = np.where(mask, s * scale, -np.inf)
    p = np.exp(z - z.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    assert (p.max(1) >= 0.4).mean() >= 0.9


@pytest.mark.parametrize("causal", [False, True])
def test_planted_list_mistakes_exceed_tolerance_1d(causal):
    n, r = 512, 32
    w, q, k, v, pk, pv = _inputs(1, causal, n, r, 21 + causal)
    scale = fma_inputs.PEAKED_SCALE
    kaug, vaug = _augmented_1d(n, r, k, v, pk, pv)
    mask = brute.mask_1d(n, r, causal)
    ref = brute.masked_attention(q, kaug, vaug, mask, scale)
    sizes, offs = _level_offsets_1d(n, r)
    moves = {}

    # a whole level dropped
    for li in range(len(sizes)):
        m = mask.copy()
        m[:, n + offs[li]:n + offs[li + 1]] = False
        moves["drop level %d" % (li + 1)] = _rel(brute.masked_attention(q, kaug, vaug, m, scale), ref)

    # list entry j of every level dropped (the closed-form slot j)
    lists, _, _ = oracle.lists_1d(n, r, kcap=3)
    for j in range(3):
        m = mask.copy()
        for i in range(n):
            for li in range(len(sizes)):
                g = lists[i // r, li, j]
                if g >= 0:
                    m[i, n + offs[li] + g] = False
        if (m != mask).any():
            moves["drop slot %d" % j] = _rel(brute.masked_attention(q, kaug, vaug, m, scale), ref)

    # the next (bidirectional) or previous near block dropped
    m = mask.copy()
    for i in range(n):
        b = i // r
        nb = b + 1 if not causal else b - 1
        if 0 <= nb < n // r:
            m[i, nb * r:(nb + 1) * r] = False
    moves["drop near block"] = _rel(brute.masked_attention(q, kaug, vaug, m, scale), ref)

    # an empty list slot read as coarse row 0 (the row an empty slot points at)
    m = mask.copy()
    for i in range(n):
        if (lists[i // r] < 0).any():
            m[i, n] = True
    if (m != mask).any():
        moves["empty slot unmasked"] = _rel(brute.masked_attention(q, kaug, vaug, m, scale), ref)

    # aggregation weights one offset off: pi shifted by one inside each level
    pk2 = np.concatenate([np.roll(pk[offs_w:offs_w + s], 1)
                          for offs_w, s in zip(np.cumsum([0] + sizes[:-1]), sizes)])
    kaug2, _ = _augmented_1d(n, r, k, v, pk2, pv)
    moves["weight offset +1"] = _rel(brute.masked_attention(q, kaug2, vaug, mask, scale), ref)

    if causal:
        # a future token of the diagonal block leaked
        m = mask.copy()
        for i in range(n - 1):
            if (i + 1) // r == i // r:
                m[i, i + 1] = True
        moves["future token leaked"] = _rel(brute.masked_attention(q, kaug, vaug, m, scale), ref)
        # the group right after the visible ones (g = q - 1) leaked
        m = mask.copy()
        for i in range(n):
            b = i // r
            for li, s in enumerate(sizes):
                g = (b >> li) - 1
                if 0 <= g < offs[li + 1] - offs[li]:
                    m[i, n + offs[li] + g] = True
        moves["non-past group leaked"] = _rel(brute.masked_attention(q, kaug, vaug, m, scale), ref)

    for what, mv in moves.items():
        assert mv >= MIN_MOVE, (what, mv)
    assert min(moves.values()) > 10 * TOL_BF16


def test_planted_list_mistakes_exceed_tolerance_2d():
    W, r = 32, 4
    w, q, k, v, pk, pv = _inputs(2, False, W, r, 31)
    n = W * W
    scale = fma_inputs.PEAKED_SCALE
    out = oracle.forward_2d(q, k, v, W, r, pk, pv, scale=scale)
    A = brute.aggregation_matrix_2d(W, r, pk)
    kaug = np.vstack([k, A @ k])
    vaug = np.vstack([v, brute.aggregation_matrix_2d(W, r, pv) @ v])
    mask = brute.mask_2d(W, r)
    ref = brute.masked_attention(q, kaug, vaug, mask, scale)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    L = oracle.num_levels(W // r)
    sizes = [r * 2 ** (l - 1) for l in range(1, L)]
    offs = np.cumsum([0] + [(-(-W // s)) ** 2 for s in sizes])
    lists = oracle.lists_2d(W, r, kcap=27)
    moves = {}
    for li in range(len(sizes)):
        m = mask.copy()
        m[:, n + offs[li]:n + offs[li + 1]] = False
        moves["drop level %d" % (li + 1)] = _rel(brute.masked_attention(q, kaug, vaug, m, scale), ref)
    # list entries of one window row (slots 0..5 of every level) dropped
    m = mask.copy()
    nbx = W // r
    for i in range(n):
        cell = (i // W // r) * nbx + (i % W) // r
        for li in range(len(sizes)):
            for j in range(6):
                g = lists[cell, li, j]
                if g >= 0:
                    m[i, n + offs[li] + g] = False
    moves["drop window row"] = _rel(brute.masked_attention(q, kaug, vaug, m, scale), ref)
    # the near cell below dropped
    m = mask.copy()
    for i in range(n):
        x, y = divmod(i, W)
        cx = x // r + 1
        if cx < nbx:
            for xx in range(cx * r, (cx + 1) * r):
                m[i, xx * W + (y // r) * r: xx * W + (y // r + 1) * r] = False
    moves["drop near cell"] = _rel(brute.masked_attention(q, kaug, vaug, m, scale), ref)
    # x and y weights swapped (transposed aggregation)
    pk2 = pk.copy()
    o = 0
    for s in sizes:
        pk2[o:o + s], pk2[o + s:o + 2 * s] = pk[o + s:o + 2 * s], pk[o:o + s]
        o += 2 * s
    kaug2 = np.vstack([k, brute.aggregation_matrix_2d(W, r, pk2) @ k])
    moves["x/y weights swapped"] = _rel(brute.masked_attention(q, kaug2, vaug, mask, scale), ref)
    for what, mv in moves.items():
        assert mv >= MIN_MOVE, (what, mv)


def test_peaked_inputs_layout_matches_make_inputs():
    """make_peaked_inputs draws weights in make_inputs' layout (per head, per
    level and basis; 2D [pi_x | pi_y]), each vector one-hot."""
    for w in (fma_inputs.custom("a", 1, True, "bf16", 2, 3, n=2048, block=64, rank=2),
              fma_inputs.custom("b", 2, False, "bf16", 1, 2, side=64, block=8, rank=3)):
        q, k, v, wk, wv = fma_inputs.make_inputs(w)
        q2, k2, v2, wk2, wv2 = fma_inputs.make_peaked_inputs(w)
        assert q2.shape == q.shape and wk2.shape == wk.shape and wv2.shape == wv.shape
        assert q2.dtype == q.dtype
        assert torch.equal(q2.float(), q2.float().round()) and q2.abs().max() <= 2
        nvec = sum(1 for _ in fma_inputs.level_sizes(w)) * w.rank * (1 if w.ndim == 1 else 2)
        assert torch.equal(wk2.sum(1), torch.full((w.heads,), float(nvec)))
        assert torch.equal((wk2 != 0).sum(1), torch.full((w.heads,), nvec))
