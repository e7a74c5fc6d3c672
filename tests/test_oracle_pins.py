"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test ties the oracle (oracle/fma_oracle.c) to something other than
itself: a library routine in a special case, a brute-force rebuild of the
index sets from the set-builder definitions, closed-form work counts, an
invariant, or the independent dense formulation in oracle/brute.py.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import brute


def _rng(seed):
    return np.random.default_rng(seed)


def _qkv(n, d, seed, lead=()):
    g = _rng(seed)
    return [g.standard_normal(lead + (n, d)) for _ in range(3)]


def _pi_1d(n, r, seed, heads=None):
    L = oracle.num_levels(n // r)
    g = _rng(seed)
    parts = [g.standard_normal(((heads or 1), r * 2 ** (l - 1))) / np.sqrt(r * 2 ** (l - 1))
             for l in range(1, L)]
    w = np.concatenate(parts, axis=1) if parts else np.zeros(((heads or 1), 0))
    return w if heads else w[0]


def _pi_2d(W, r, seed):
    L = oracle.num_levels(W // r)
    g = _rng(seed)
    parts = []
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        parts += [g.standard_normal(s) / np.sqrt(s), g.standard_normal(s) / np.sqrt(s)]
    return np.concatenate(parts) if parts else np.zeros(0)


def _closed_form_1d(n, r, b, l, causal=False):
    """Interaction list of base block b at level l: the level-l groups in the
    6-group window of the parent pair, minus the 3 groups around q."""
    s = r * 2 ** (l - 1)
    M = -(-n // s)
    q = b >> (l - 1)
    p = q >> 1
    out = [g for g in range(2 * p - 2, 2 * p + 4) if 0 <= g < M and abs(g - q) > 1]
    if causal:
        out = [g for g in out if g <= q - 2]
    return out


# ------------------------------------------------------------------ pin 1
@pytest.mark.parametrize("n,r", [(64, 64), (128, 64), (96, 48), (16, 8), (6, 3)])
@pytest.mark.parametrize("causal", [False, True])
def test_degenerate_hierarchy_is_dense_attention(n, r, causal):
    """With one or two base blocks the near field is the whole sequence and
    FMA is softmax(QK^T/sqrt(d))V (Sec. 1, Eq. attn)."""
    q, k, v = _qkv(n, 16, 1 + n + r)
    out = oracle.forward_1d(q, k, v, r, causal=causal)
    t = lambda a: torch.from_numpy(a)[None, None]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=causal)
    np.testing.assert_allclose(out, ref[0, 0].numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("W,r", [(8, 8), (8, 4), (6, 3)])
def test_degenerate_hierarchy_is_dense_attention_2d(W, r):
    q, k, v = _qkv(W * W, 8, W + r)
    out = oracle.forward_2d(q, k, v, W, r)
    t = lambda a: torch.from_numpy(a)[None, None]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v))
    np.testing.assert_allclose(out, ref[0, 0].numpy(), rtol=0, atol=1e-12)


# ------------------------------------------------------------------ pin 2/3
@pytest.mark.parametrize("nb", list(range(1, 40)))
@pytest.mark.parametrize("r", [1, 2, 3])
def test_sets_1d_brute_force_and_closed_form(nb, r):
    """Set-builder export == per-row brute force == closed form, and the near
    and far sets of every row form a disjoint cover of [n]."""
    n = nb * r
    L = oracle.num_levels(nb)
    lists, lo, hi = oracle.lists_1d(n, r, kcap=3)
    for i in range(n):
        b = i // r
        near, far = brute.sets_row_1d(n, r, i)
        assert near == list(range(lo[b], hi[b]))
        lab = oracle.labels_1d(n, r, i)
        assert sorted(np.flatnonzero(lab == 0).tolist()) == near
        covered = list(near)
        for l in range(1, L):
            got = [g for g in lists[b, l - 1].tolist() if g >= 0]
            assert got == far[l], (n, r, i, l)
            assert got == _closed_form_1d(n, r, b, l)
            s = r * 2 ** (l - 1)
            toks = [j for m in got for j in range(m * s, min((m + 1) * s, n))]
            assert sorted(toks) == sorted(np.flatnonzero(lab == l).tolist())
            covered += toks
        assert sorted(covered) == list(range(n))  # disjoint (no repeats) cover


@pytest.mark.parametrize("W,r", [(4, 1), (6, 1), (8, 1), (10, 1), (12, 1), (16, 1),
                                 (8, 2), (12, 2), (16, 2), (6, 2)])
def test_sets_2d_brute_force_and_closed_form(W, r):
    nbx = W // r
    L = oracle.num_levels(nbx)
    lists = oracle.lists_2d(W, r, kcap=27)
    for i in range(W * W):
        x, y = divmod(i, W)
        cell = (x // r) * nbx + (y // r)
        near, far = brute.sets_row_2d(W, r, i)
        lab = oracle.labels_2d(W, r, i)
        assert sorted(np.flatnonzero(lab == 0).tolist()) == near
        covered = list(near)
        for l in range(1, L):
            s = r * 2 ** (l - 1)
            M = -(-W // s)
            got = [g for g in lists[cell, l - 1].tolist() if g >= 0]
            assert got == far[l], (W, r, i, l)
            qx, qy = (x // r) >> (l - 1), (y // r) >> (l - 1)
            px, py = qx >> 1, qy >> 1
            closed = [u * M + v for u in range(2 * px - 2, 2 * px + 4)
                      for v in range(2 * py - 2, 2 * py + 4)
                      if 0 <= u < M and 0 <= v < M and not (abs(u - qx) <= 1 and abs(v - qy) <= 1)]
            assert got == closed
            pix = [xx * W + yy for g in got for xx in range((g // M) * s, min((g // M + 1) * s, W))
                   for yy in range((g % M) * s, min((g % M + 1) * s, W))]
            assert sorted(pix) == sorted(np.flatnonzero(lab == l).tolist())
            covered += pix
        assert sorted(covered) == list(range(W * W))


def test_causal_rule_equals_closed_form():
    """A far group is visible to row i iff all its tokens are <= i; for the
    groups of the interaction list that is g <= q - 2."""
    for nb in range(1, 33):
        for r in (1, 2, 4):
            n = nb * r
            L = oracle.num_levels(nb)
            for i in range(n):
                b = i // r
                _, far = brute.sets_row_1d(n, r, i)
                for l in range(1, L):
                    s = r * 2 ** (l - 1)
                    vis = [m for m in far[l] if min((m + 1) * s, n) - 1 <= i]
                    assert vis == _closed_form_1d(n, r, b, l, causal=True)


# ------------------------------------------------------------------ pin 4
@pytest.mark.parametrize("r", [1, 2, 4, 8])
@pytest.mark.parametrize("L", [2, 3, 4, 5, 6])
def test_work_counts_1d(r, L):
    """Sources per row: near <= 3r, plus 3 groups per level (Sec. 3: at most
    3r + O(log n) sources); totals O(n log n); coarse rows 2n/r - 4 = O(n)."""
    n = r * 2 ** L
    q, k, v = _qkv(n, 4, 7)
    pk, pv = _pi_1d(n, r, 8), _pi_1d(n, r, 9)
    _, cb = oracle.forward_1d(q, k, v, r, pk, pv, causal=False, return_counts=True)
    _, cc = oracle.forward_1d(q, k, v, r, pk, pv, causal=True, return_counts=True)
    near_b = r * (3 * n - 2 * r)
    near_c = r * (n - r) + n * (r + 1) // 2
    far_b = (3 * n * (L - 2) + 6 * r) if L >= 2 else 0
    assert cb.sum() == near_b + far_b
    assert 2 * (cc.sum() - near_c) == far_b
    assert cb.max() <= 3 * r + 3 * (L - 1)
    assert cc.max() <= 2 * r + 2 * (L - 1)
    assert oracle.coarse_rows_1d(n, r) == (2 * n // r - 4 if L >= 2 else 0)


@pytest.mark.parametrize("W,r", [(16, 2), (16, 1), (32, 2), (32, 4)])
def test_work_counts_2d(W, r):
    """Sources per pixel: at most 9 r^2 near + 27 per level (Sec. 3)."""
    M0 = W // r
    L = oracle.num_levels(M0)
    q, k, v = _qkv(W * W, 2, 3)
    pk, pv = _pi_2d(W, r, 4), _pi_2d(W, r, 5)
    _, c = oracle.forward_2d(q, k, v, W, r, pk, pv, return_counts=True)
    near = r ** 4 * (3 * M0 - 2) ** 2
    far = 0
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        M = W // s
        far += s * s * ((6 * M - 8) ** 2 - (3 * M - 2) ** 2)
    assert c.sum() == near + far
    assert c.max() <= 9 * r * r + 27 * (L - 1)


# ------------------------------------------------------------------ pin 5
def test_stencil_tiers():
    """Fig. 1: beyond the 3r near window the tiers merge r, 2r, 4r tokens;
    2D: the first coarse tier of an interior cell holds 6x6 - 3x3 = 27
    squares (the isotropic 3x3 stencil of Sec. 2)."""
    n, r = 64 * 4, 4
    i = n // 2
    _, far = brute.sets_row_1d(n, r, i)
    for l in (1, 2, 3):
        assert len(far[l]) == 3
    lists, _, _ = oracle.lists_1d(n, r)
    sizes = {l: r * 2 ** (l - 1) for l in (1, 2, 3)}
    assert sizes == {1: r, 2: 2 * r, 3: 4 * r}
    W, r2 = 32, 2
    cell = (W // r2 // 2) * (W // r2) + W // r2 // 2
    l2 = oracle.lists_2d(W, r2)
    assert (l2[cell, 0] >= 0).sum() == 27


# ------------------------------------------------------------------ pin 6
@pytest.mark.parametrize("n,r,causal", [(256, 8, False), (256, 8, True), (96, 8, False),
                                        (120, 8, True)])
def test_joint_weights_sum_to_one(n, r, causal):
    """V = 1 and pi^v_l = 1/s_l make every coarse value 1; a convex
    combination of ones is one."""
    q, k, _ = _qkv(n, 8, 11)
    L = oracle.num_levels(n // r)
    v = np.ones((n, 8))
    pk = _pi_1d(n, r, 12)
    pv = np.concatenate([np.full(r * 2 ** (l - 1), 1.0 / (r * 2 ** (l - 1))) for l in range(1, L)])
    out = oracle.forward_1d(q, k, v, r, pk, pv, causal=causal)
    np.testing.assert_allclose(out, 1.0, rtol=0, atol=1e-12)
    # the printed per-set normalisation sums to 1 + (number of non-empty levels)
    out2 = oracle.forward_1d(q, k, v, r, pk, pv, causal=causal, norm=oracle.NORM_PER_SET)
    for i in range(n):
        _, far = brute.sets_row_1d(n, r, i)
        nonempty = 0
        for l, G in far.items():
            s = r * 2 ** (l - 1)
            vis = [m for m in G if not causal or min((m + 1) * s, n) - 1 <= i]
            nonempty += bool(vis)
        np.testing.assert_allclose(out2[i], 1.0 + nonempty, rtol=0, atol=1e-12)


def test_joint_weights_sum_to_one_2d():
    W, r = 16, 2
    q, k, _ = _qkv(W * W, 8, 13)
    L = oracle.num_levels(W // r)
    v = np.ones((W * W, 8))
    pk = _pi_2d(W, r, 14)
    pv = np.concatenate([np.full(2 * r * 2 ** (l - 1), 1.0 / (r * 2 ** (l - 1))) for l in range(1, L)])
    out = oracle.forward_2d(q, k, v, W, r, pk, pv)
    np.testing.assert_allclose(out, 1.0, rtol=0, atol=1e-12)


# ------------------------------------------------------------------ pin 7
@pytest.mark.parametrize("n,r", [(256, 8), (192, 16), (104, 8)])
def test_causality(n, r):
    """Changing tokens after t leaves every row <= t unchanged, bit for bit."""
    q, k, v = _qkv(n, 8, 21)
    pk, pv = _pi_1d(n, r, 22), _pi_1d(n, r, 23)
    base = oracle.forward_1d(q, k, v, r, pk, pv, causal=True)
    g = _rng(24)
    for t in (0, r - 1, r, n // 2 + 3, n - 2):
        q2, k2, v2 = q.copy(), k.copy(), v.copy()
        for a in (q2, k2, v2):
            a[t + 1:] = g.standard_normal(a[t + 1:].shape) * 5
        out = oracle.forward_1d(q2, k2, v2, r, pk, pv, causal=True)
        assert np.array_equal(out[:t + 1], base[:t + 1])
        assert not np.array_equal(out[t + 1:], base[t + 1:])


# ------------------------------------------------------------------ pin 8
@pytest.mark.parametrize("n,r", [(256, 8), (512, 16)])
def test_reversal_equivariance(n, r):
    """Bidirectional 1D with n/r a power of two: reversing the sequence and
    every level's weight vector reverses the output."""
    q, k, v = _qkv(n, 8, 31)
    L = oracle.num_levels(n // r)
    pk, pv = _pi_1d(n, r, 32), _pi_1d(n, r, 33)

    def rev_levels(p):
        out, off = [], 0
        for l in range(1, L):
            s = r * 2 ** (l - 1)
            out.append(p[off:off + s][::-1])
            off += s
        return np.concatenate(out)

    a = oracle.forward_1d(q, k, v, r, pk, pv)
    b = oracle.forward_1d(q[::-1], k[::-1], v[::-1], r, rev_levels(pk), rev_levels(pv))
    np.testing.assert_allclose(b[::-1], a, rtol=0, atol=1e-12)


def test_transpose_equivariance_2d():
    """Transposing the map and swapping pi^(x) with pi^(y) transposes the output."""
    W, r, d = 16, 2, 8
    q, k, v = _qkv(W * W, d, 41)
    L = oracle.num_levels(W // r)
    pk, pv = _pi_2d(W, r, 42), _pi_2d(W, r, 43)

    def swap(p):
        out, off = [], 0
        for l in range(1, L):
            s = r * 2 ** (l - 1)
            out += [p[off + s:off + 2 * s], p[off:off + s]]
            off += 2 * s
        return np.concatenate(out)

    T = lambda a: a.reshape(W, W, d).transpose(1, 0, 2).reshape(W * W, d)
    a = oracle.forward_2d(q, k, v, W, r, pk, pv)
    b = oracle.forward_2d(T(q), T(k), T(v), W, r, swap(pk), swap(pv))
    np.testing.assert_allclose(T(b), a, rtol=0, atol=1e-12)


# ------------------------------------------------------------------ pin 9
@pytest.mark.parametrize("n,r,causal", [(128, 8, False), (128, 8, True), (96, 8, False),
                                        (88, 8, True), (64, 4, False), (40, 4, True)])
def test_dense_masked_formulation_1d(n, r, causal):
    """The per-row oracle equals an explicit n x (n+R) masked score matrix
    over augmented keys [K; K_bar] (independent code), and x_hat = A V for
    the effective hierarchical matrix A."""
    q, k, v = _qkv(n, 8, 51)
    pk, pv = _pi_1d(n, r, 52), _pi_1d(n, r, 53)
    out = oracle.forward_1d(q, k, v, r, pk, pv, causal=causal)
    ref = brute.forward_dense_1d(q, k, v, r, pk, pv, causal=causal)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    A = brute.hmatrix_1d(q, k, r, pk, pv, causal=causal)
    np.testing.assert_allclose(out, A @ v, rtol=0, atol=1e-12)


@pytest.mark.parametrize("W,r", [(16, 2), (12, 2), (8, 1)])
def test_dense_masked_formulation_2d(W, r):
    q, k, v = _qkv(W * W, 8, 61)
    pk, pv = _pi_2d(W, r, 62), _pi_2d(W, r, 63)
    out = oracle.forward_2d(q, k, v, W, r, pk, pv)
    ref = brute.forward_dense_2d(q, k, v, W, r, pk, pv)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_batched_heads_match_slices():
    """Per-head weights apply to their own head in every batch entry."""
    B, H, n, r, d = 2, 3, 64, 8, 4
    g = _rng(71)
    q, k, v = [g.standard_normal((B, H, n, d)) for _ in range(3)]
    pk, pv = _pi_1d(n, r, 72, heads=H), _pi_1d(n, r, 73, heads=H)
    out = oracle.forward_1d(q, k, v, r, pk, pv)
    for b in range(B):
        for h in range(H):
            ref = brute.forward_dense_1d(q[b, h], k[b, h], v[b, h], r, pk[h], pv[h])
            np.testing.assert_allclose(out[b, h], ref, rtol=0, atol=1e-12)


# ------------------------------------------------------------------ pin 10
def test_coarsening_special_cases_1d():
    n, r, d = 256, 8, 5
    g = _rng(81)
    x = g.standard_normal((n, d))
    L = oracle.num_levels(n // r)
    # one-hot weight at offset o picks token g*s + o
    for o in (0, 3, 7):
        pi = np.concatenate([np.eye(r * 2 ** (l - 1))[o] for l in range(1, L)])
        out = oracle.coarsen_1d(x, r, pi)
        row = 0
        for l in range(1, L):
            s = r * 2 ** (l - 1)
            for m in range(n // s):
                assert np.array_equal(out[row], x[m * s + o])
                row += 1
    # uniform weights are average pooling
    pi = np.concatenate([np.full(r * 2 ** (l - 1), 1.0 / (r * 2 ** (l - 1))) for l in range(1, L)])
    out = oracle.coarsen_1d(x, r, pi)
    row = 0
    xt = torch.from_numpy(x.T.copy())[None]
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        pooled = torch.nn.functional.avg_pool1d(xt, s, s)[0].T.numpy()
        np.testing.assert_allclose(out[row:row + n // s], pooled, rtol=1e-13, atol=1e-14)
        row += n // s
    # random weights agree with the dense aggregation matrix
    pi = _pi_1d(n, r, 82)
    np.testing.assert_allclose(oracle.coarsen_1d(x, r, pi),
                               brute.aggregation_matrix_1d(n, r, pi) @ x, rtol=1e-12, atol=1e-13)


def test_coarsening_ragged_tail_1d():
    """n/r not a power of two: the last group of a level is clipped to [n]."""
    n, r, d = 88, 8, 3
    x = _rng(83).standard_normal((n, d))
    pi = _pi_1d(n, r, 84)
    np.testing.assert_allclose(oracle.coarsen_1d(x, r, pi),
                               brute.aggregation_matrix_1d(n, r, pi) @ x, rtol=1e-12, atol=1e-13)


def test_coarsening_special_cases_2d():
    W, r, d = 16, 2, 3
    g = _rng(85)
    x = g.standard_normal((W * W, d))
    L = oracle.num_levels(W // r)
    a0, b0 = 1, 0
    pi = np.concatenate([np.concatenate([np.eye(r * 2 ** (l - 1))[a0], np.eye(r * 2 ** (l - 1))[b0]])
                         for l in range(1, L)])
    out = oracle.coarsen_2d(x, W, r, pi)
    row = 0
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        M = W // s
        for u in range(M):
            for v in range(M):
                assert np.array_equal(out[row], x[(u * s + a0) * W + v * s + b0])
                row += 1
    # uniform weights: 2D average pooling
    pi = np.concatenate([np.full(2 * r * 2 ** (l - 1), 1.0 / (r * 2 ** (l - 1))) for l in range(1, L)])
    out = oracle.coarsen_2d(x, W, r, pi)
    img = torch.from_numpy(x.T.reshape(d, W, W).copy())[None]
    row = 0
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        M = W // s
        pooled = torch.nn.functional.avg_pool2d(img, s, s)[0].reshape(d, M * M).T.numpy()
        np.testing.assert_allclose(out[row:row + M * M], pooled, rtol=1e-13, atol=1e-14)
        row += M * M
    # the direct double sum equals the separable two-pass form
    pi = _pi_2d(W, r, 86)
    out = oracle.coarsen_2d(x, W, r, pi)
    img = x.reshape(W, W, d)
    row, off = 0, 0
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        px, py = pi[off:off + s], pi[off + s:off + 2 * s]
        off += 2 * s
        M = W // s
        t = np.einsum("xvbc,b->xvc", img.reshape(W, M, s, d), py)       # along y
        sep = np.einsum("uavc,a->uvc", t.reshape(M, s, M, d), px)      # along x
        np.testing.assert_allclose(out[row:row + M * M], sep.reshape(M * M, d), rtol=1e-12, atol=1e-13)
        row += M * M


# ------------------------------------------------------------------ pin 11
def test_linearity_in_values():
    n, r = 128, 8
    q, k, v1 = _qkv(n, 8, 91)
    v2 = _rng(92).standard_normal((n, 8))
    pk, pv = _pi_1d(n, r, 93), _pi_1d(n, r, 94)
    a, b = 0.7, -1.9
    lhs = oracle.forward_1d(q, k, a * v1 + b * v2, r, pk, pv, causal=True)
    rhs = a * oracle.forward_1d(q, k, v1, r, pk, pv, causal=True) + \
        b * oracle.forward_1d(q, k, v2, r, pk, pv, causal=True)
    np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-12)


def test_oracle_rejects_bad_shapes():
    q, k, v = _qkv(100, 4, 1)
    with pytest.raises(RuntimeError):
        oracle.forward_1d(q, k, v, 8)          # 8 does not divide 100


# ------------------------------------------------------------------ pin 12
# Coarse level rank p (Sec. 3): p basis vectors per level, p aggregated keys
# and values per group, every representative a source of its own.
def _pi_rank_1d(n, r, p, seed):
    L = oracle.num_levels(n // r)
    g = _rng(seed)
    parts = [g.standard_normal(r * 2 ** (l - 1)) / np.sqrt(r * 2 ** (l - 1))
             for l in range(1, L) for _ in range(p)]
    return np.concatenate(parts) if parts else np.zeros(0)


def _pi_rank_2d(W, r, p, seed):
    L = oracle.num_levels(W // r)
    g = _rng(seed)
    parts = [g.standard_normal(2 * r * 2 ** (l - 1)) / np.sqrt(r * 2 ** (l - 1))
             for l in range(1, L) for _ in range(p)]
    return np.concatenate(parts) if parts else np.zeros(0)


def _repeat_bases(pi, sizes, p):
    """Rank-1 weights -> rank-p weights whose p bases per level are equal."""
    out, off = [], 0
    for s in sizes:
        out += [pi[off:off + s]] * p
        off += s
    return np.concatenate(out) if out else np.zeros(0)


@pytest.mark.parametrize("n,r,causal,p", [(128, 8, False, 2), (128, 8, True, 3), (88, 8, True, 2),
                                          (64, 4, False, 4), (40, 4, True, 3), (256, 16, True, 4)])
def test_rank_p_dense_formulation_1d(n, r, causal, p):
    """Group-major per-row sources (C oracle) equal a dense masked softmax
    whose coarse columns are repeated basis-major (independent code)."""
    q, k, v = _qkv(n, 8, 121)
    pk, pv = _pi_rank_1d(n, r, p, 122), _pi_rank_1d(n, r, p, 123)
    out = oracle.forward_1d(q, k, v, r, pk, pv, causal=causal, rank=p)
    ref = brute.forward_dense_1d(q, k, v, r, pk, pv, causal=causal, rank=p)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("W,r,p", [(16, 2, 2), (12, 2, 3), (8, 1, 4)])
def test_rank_p_dense_formulation_2d(W, r, p):
    q, k, v = _qkv(W * W, 8, 124)
    pk, pv = _pi_rank_2d(W, r, p, 125), _pi_rank_2d(W, r, p, 126)
    out = oracle.forward_2d(q, k, v, W, r, pk, pv, rank=p)
    ref = brute.forward_dense_2d(q, k, v, W, r, pk, pv, rank=p)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("p", [2, 3])
def test_rank_p_identical_bases(causal, p):
    """p equal bases put every group in the joint softmax p times: the same
    as rank 1 with every coarse logit raised by log p.  Under the per-set
    normalisation the p copies cancel and rank 1 comes back exactly."""
    n, r, d = 128, 8, 8
    q, k, v = _qkv(n, d, 127)
    L = oracle.num_levels(n // r)
    sizes = [r * 2 ** (l - 1) for l in range(1, L)]
    pk, pv = _pi_1d(n, r, 128), _pi_1d(n, r, 129)
    pkp, pvp = _repeat_bases(pk, sizes, p), _repeat_bases(pv, sizes, p)
    out = oracle.forward_1d(q, k, v, r, pkp, pvp, causal=causal, rank=p)
    # closed form: softmax over [K; K_bar] with log p added to coarse logits
    scale = 1.0 / np.sqrt(d)
    mask = brute.mask_1d(n, r, causal)
    kaug = np.vstack([k, brute.aggregation_matrix_1d(n, r, pk) @ k])
    vaug = np.vstack([v, brute.aggregation_matrix_1d(n, r, pv) @ v])
    s = scale * q @ kaug.T
    s[:, n:] += np.log(p)
    s = np.where(mask, s, -np.inf)
    w = np.exp(s - s.max(axis=1, keepdims=True))
    ref = (w / w.sum(axis=1, keepdims=True)) @ vaug
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    # per-set normalisation: identical copies leave each level's weights as at rank 1
    a = oracle.forward_1d(q, k, v, r, pkp, pvp, causal=causal, rank=p, norm=oracle.NORM_PER_SET)
    b = oracle.forward_1d(q, k, v, r, pk, pv, causal=causal, norm=oracle.NORM_PER_SET)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_rank_p_identical_bases_2d():
    W, r, p, d = 16, 2, 3, 8
    q, k, v = _qkv(W * W, d, 130)
    L = oracle.num_levels(W // r)
    sizes = [2 * r * 2 ** (l - 1) for l in range(1, L)]
    pk, pv = _pi_2d(W, r, 131), _pi_2d(W, r, 132)
    out = oracle.forward_2d(q, k, v, W, r, _repeat_bases(pk, sizes, p), _repeat_bases(pv, sizes, p),
                            rank=p)
    scale = 1.0 / np.sqrt(d)
    mask = brute.mask_2d(W, r)
    kaug = np.vstack([k, brute.aggregation_matrix_2d(W, r, pk) @ k])
    vaug = np.vstack([v, brute.aggregation_matrix_2d(W, r, pv) @ v])
    s = scale * q @ kaug.T
    s[:, W * W:] += np.log(p)
    s = np.where(mask, s, -np.inf)
    w = np.exp(s - s.max(axis=1, keepdims=True))
    np.testing.assert_allclose(out, (w / w.sum(axis=1, keepdims=True)) @ vaug, rtol=0, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_rank_p_work_counts(causal):
    """Every far group contributes p sources, the near field is unchanged."""
    n, r, p = 256, 8, 4
    q, k, v = _qkv(n, 4, 133)
    _, c1 = oracle.forward_1d(q, k, v, r, _pi_1d(n, r, 134), _pi_1d(n, r, 135), causal=causal,
                              return_counts=True)
    _, cp = oracle.forward_1d(q, k, v, r, _pi_rank_1d(n, r, p, 136), _pi_rank_1d(n, r, p, 137),
                              causal=causal, return_counts=True, rank=p)
    for i in range(n):
        near, _ = brute.sets_row_1d(n, r, i)
        nn = sum(1 for j in near if not causal or j <= i)
        assert cp[i] - nn == p * (c1[i] - nn)


def test_rank_p_coarsening():
    """Rows are (level, basis, group); basis b of level l aggregates with its
    own weights.  One-hot bases pick distinct tokens exactly."""
    n, r, p, d = 88, 8, 3, 5
    g = _rng(138)
    x = g.standard_normal((n, d))
    L = oracle.num_levels(n // r)
    pi = _pi_rank_1d(n, r, p, 139)
    out = oracle.coarsen_1d(x, r, pi, rank=p)
    per_basis = [brute.aggregation_matrix_1d(n, r, w) @ x for w in brute.rank_bases_1d(n, r, pi, p)]
    off = 0
    for l in range(1, L):
        M = -(-n // (r * 2 ** (l - 1)))
        for m in range(M):
            for b in range(p):
                np.testing.assert_allclose(out[p * off + b * M + m], per_basis[b][off + m],
                                           rtol=1e-12, atol=1e-13)
        off += M
    assert out.shape[0] == p * off
    # one-hot bases at offsets 0, 1, 2
    n = 128
    x = g.standard_normal((n, d))
    L = oracle.num_levels(n // r)
    pi = np.concatenate([np.eye(r * 2 ** (l - 1))[b] for l in range(1, L) for b in range(p)])
    out = oracle.coarsen_1d(x, r, pi, rank=p)
    row = 0
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        for b in range(p):
            for m in range(n // s):
                assert np.array_equal(out[row], x[m * s + b])
                row += 1


def test_rank_p_coarsening_2d():
    W, r, p, d = 12, 2, 2, 3
    x = _rng(140).standard_normal((W * W, d))
    L = oracle.num_levels(W // r)
    pi = _pi_rank_2d(W, r, p, 141)
    out = oracle.coarsen_2d(x, W, r, pi, rank=p)
    per_basis = [brute.aggregation_matrix_2d(W, r, w) @ x for w in brute.rank_bases_2d(W, r, pi, p)]
    off = 0
    for l in range(1, L):
        MM = (-(-W // (r * 2 ** (l - 1)))) ** 2
        for gsq in range(MM):
            for b in range(p):
                np.testing.assert_allclose(out[p * off + b * MM + gsq], per_basis[b][off + gsq],
                                           rtol=1e-12, atol=1e-13)
        off += MM


def test_rank_p_rejects_wrong_weight_length():
    n, r = 64, 8
    q, k, v = _qkv(n, 4, 142)
    with pytest.raises(ValueError):
        oracle.forward_1d(q, k, v, r, _pi_1d(n, r, 1), _pi_1d(n, r, 2), rank=2)


# ------------------------------------------------------------------ pin 13
# The printed normalisation (Eq. fma1d / Eq. fma2d as printed): alpha over the
# near field, each beta^l over its level's groups (all p representatives).
@pytest.mark.parametrize("n,r,causal,p", [(128, 8, False, 1), (128, 8, True, 1), (88, 8, True, 1),
                                          (64, 4, False, 3), (128, 8, True, 4), (40, 4, False, 2)])
def test_per_level_dense_formulation_1d(n, r, causal, p):
    q, k, v = _qkv(n, 8, 151)
    pk, pv = _pi_rank_1d(n, r, p, 152), _pi_rank_1d(n, r, p, 153)
    out = oracle.forward_1d(q, k, v, r, pk, pv, causal=causal, rank=p, norm=oracle.NORM_PER_SET)
    ref = brute.forward_dense_1d(q, k, v, r, pk, pv, causal=causal, rank=p, per_level=True)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("W,r,p", [(16, 2, 1), (12, 2, 1), (8, 1, 2)])
def test_per_level_dense_formulation_2d(W, r, p):
    q, k, v = _qkv(W * W, 8, 154)
    pk, pv = _pi_rank_2d(W, r, p, 155), _pi_rank_2d(W, r, p, 156)
    out = oracle.forward_2d(q, k, v, W, r, pk, pv, rank=p, norm=oracle.NORM_PER_SET)
    ref = brute.forward_dense_2d(q, k, v, W, r, pk, pv, rank=p, per_level=True)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_per_level_single_level_is_two_softmaxes():
    """With one coarse level (n = 4r) the printed form is dense softmax over
    the near tokens plus a separate softmax over the visible groups."""
    n, r, d = 32, 8, 4
    q, k, v = _qkv(n, d, 157)
    pk, pv = _pi_1d(n, r, 158), _pi_1d(n, r, 159)
    out = oracle.forward_1d(q, k, v, r, pk, pv, norm=oracle.NORM_PER_SET)
    kb, vb = oracle.coarsen_1d(k, r, pk), oracle.coarsen_1d(v, r, pv)   # 4 groups of 8
    tau = 1.0 / np.sqrt(d)
    for i in range(n):
        b = i // r
        near = [j for j in range(n) if abs(j // r - b) <= 1]
        far = [g for g in range(4) if abs(g - b) > 1]
        sn = torch.softmax(torch.tensor(tau * q[i] @ k[near].T), 0).numpy()
        ref = sn @ v[near]
        if far:
            sf = torch.softmax(torch.tensor(tau * q[i] @ kb[far].T), 0).numpy()
            ref = ref + sf @ vb[far]
        np.testing.assert_allclose(out[i], ref, rtol=0, atol=1e-12)


# ------------------------------------------------------------------ pin 14
# Backward (gradients for end-to-end training of the weights).
def _grads_torch(q, k, v, r, pk, pv, dout, causal=False, rank=1, per_level=False, W=None):
    T = [torch.tensor(x, requires_grad=True) for x in (q, k, v, pk, pv)]
    out = brute.forward_torch(*T[:3], r, T[3], T[4], causal=causal, rank=rank, per_level=per_level, W=W)
    (out * torch.tensor(dout)).sum().backward()
    return [t.grad.numpy() for t in T]


@pytest.mark.parametrize("n,r,causal,p,pl", [(64, 8, False, 1, False), (64, 8, True, 1, False),
                                             (40, 4, True, 2, False), (32, 4, False, 3, False),
                                             (64, 8, True, 2, True), (48, 4, False, 1, True)])
def test_backward_matches_autograd_1d(n, r, causal, p, pl):
    """Oracle gradients = torch autograd of the independent dense formulation
    (aggregation matrices built from the weight tensors by indexing)."""
    q, k, v = _qkv(n, 6, 161)
    dout = _rng(162).standard_normal((n, 6))
    pk, pv = _pi_rank_1d(n, r, p, 163), _pi_rank_1d(n, r, p, 164)
    got = oracle.backward_1d(q, k, v, r, pk, pv, dout, causal=causal, rank=p, norm=int(pl))
    ref = _grads_torch(q, k, v, r, pk, pv, dout, causal=causal, rank=p, per_level=pl)
    for g_, r_ in zip(got, ref):
        np.testing.assert_allclose(g_, r_, rtol=0, atol=1e-12)


@pytest.mark.parametrize("W,r,p,pl", [(8, 2, 1, False), (8, 1, 2, False), (12, 2, 1, True), (8, 2, 2, True)])
def test_backward_matches_autograd_2d(W, r, p, pl):
    q, k, v = _qkv(W * W, 6, 165)
    dout = _rng(166).standard_normal((W * W, 6))
    pk, pv = _pi_rank_2d(W, r, p, 167), _pi_rank_2d(W, r, p, 168)
    got = oracle.backward_2d(q, k, v, W, r, pk, pv, dout, rank=p, norm=int(pl))
    ref = _grads_torch(q, k, v, r, pk, pv, dout, rank=p, per_level=pl, W=W)
    for g_, r_ in zip(got, ref):
        np.testing.assert_allclose(g_, r_, rtol=0, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_backward_finite_differences(causal):
    """Central differences of the (pinned) forward oracle, every input."""
    n, r, d, p = 32, 4, 4, 2
    q, k, v = _qkv(n, d, 169)
    dout = _rng(170).standard_normal((n, d))
    pk, pv = _pi_rank_1d(n, r, p, 171), _pi_rank_1d(n, r, p, 172)
    got = oracle.backward_1d(q, k, v, r, pk, pv, dout, causal=causal, rank=p)

    def loss(*a):
        return float((dout * oracle.forward_1d(*a[:3], r, a[3], a[4], causal=causal, rank=p)).sum())

    g = _rng(173)
    h = 1e-6
    for which in range(5):
        arrs = [q, k, v, pk, pv]
        for flat in g.choice(arrs[which].size, 5, replace=False):
            ix = np.unravel_index(flat, arrs[which].shape)
            plus = [a.copy() for a in arrs]
            minus = [a.copy() for a in arrs]
            plus[which][ix] += h
            minus[which][ix] -= h
            fd = (loss(*plus) - loss(*minus)) / (2 * h)
            assert abs(fd - got[which][ix]) <= 1e-6 * max(1.0, abs(fd)), (which, ix, fd, got[which][ix])


@pytest.mark.parametrize("causal", [False, True])
def test_backward_single_block_is_sdpa_backward(causal):
    """n = r: FMA is dense softmax attention, so its gradients are the
    library's attention gradients."""
    n = r = 16
    d = 8
    q, k, v = _qkv(n, d, 174)
    dout = _rng(175).standard_normal((n, d))
    got = oracle.backward_1d(q, k, v, r, None, None, dout, causal=causal)
    T = [torch.tensor(x, requires_grad=True) for x in (q, k, v)]
    out = torch.nn.functional.scaled_dot_product_attention(T[0][None], T[1][None], T[2][None], is_causal=causal)[0]
    (out * torch.tensor(dout)).sum().backward()
    for g_, t in zip(got[:3], T):
        np.testing.assert_allclose(g_, t.grad.numpy(), rtol=0, atol=1e-12)
    assert got[3] is None and got[4] is None


def test_backward_batched_weight_gradients_sum_over_batch():
    """Per-head weights collect the gradient of every batch entry of their
    head; shared weights collect every slice."""
    B, H, n, r, d = 2, 3, 32, 4, 4
    g = _rng(176)
    q, k, v, dout = [g.standard_normal((B, H, n, d)) for _ in range(4)]
    pk, pv = _pi_1d(n, r, 177, heads=H), _pi_1d(n, r, 178, heads=H)
    _, _, _, dk_, dv_ = oracle.backward_1d(q, k, v, r, pk, pv, dout)
    for h in range(H):
        acc_k = sum(oracle.backward_1d(q[b, h], k[b, h], v[b, h], r, pk[h], pv[h], dout[b, h])[3] for b in range(B))
        np.testing.assert_allclose(dk_[h], acc_k, rtol=1e-12, atol=1e-12)
    _, _, _, dks, _ = oracle.backward_1d(q, k, v, r, pk[0], pv[0], dout)
    acc = sum(oracle.backward_1d(q[b, h], k[b, h], v[b, h], r, pk[0], pv[0], dout[b, h])[3]
              for b in range(B) for h in range(H))
    np.testing.assert_allclose(dks, acc, rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------------ pin 15
# FMA-linear (query downsampling): far groups scored with the coarse query of
# the row's own group at that level.
@pytest.mark.parametrize("n,r", [(128, 8), (88, 8), (64, 4)])
def test_linear_dense_formulation_1d(n, r):
    q, k, v = _qkv(n, 8, 181)
    pk, pv, pq = _pi_1d(n, r, 182), _pi_1d(n, r, 183), _pi_1d(n, r, 184)
    out = oracle.forward_1d(q, k, v, r, pk, pv, piq=pq)
    ref = brute.forward_dense_1d(q, k, v, r, pk, pv, piq=pq)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("W,r", [(16, 2), (12, 2), (8, 1)])
def test_linear_dense_formulation_2d(W, r):
    q, k, v = _qkv(W * W, 8, 185)
    pk, pv, pq = _pi_2d(W, r, 186), _pi_2d(W, r, 187), _pi_2d(W, r, 188)
    out = oracle.forward_2d(q, k, v, W, r, pk, pv, piq=pq)
    ref = brute.forward_dense_2d(q, k, v, W, r, pk, pv, piq=pq)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_linear_constant_queries_is_fma():
    """Equal queries and query weights summing to 1 per level make every
    coarse query the token query itself: FMA-linear = FMA."""
    n, r, d = 128, 8, 8
    _, k, v = _qkv(n, d, 189)
    q = np.tile(_rng(190).standard_normal(d), (n, 1))
    L = oracle.num_levels(n // r)
    pq = np.concatenate([_rng(191 + l).dirichlet(np.ones(r * 2 ** (l - 1))) for l in range(1, L)])
    pk, pv = _pi_1d(n, r, 192), _pi_1d(n, r, 193)
    np.testing.assert_allclose(oracle.forward_1d(q, k, v, r, pk, pv, piq=pq),
                               oracle.forward_1d(q, k, v, r, pk, pv), rtol=0, atol=1e-12)
    W = 16
    _, k2, v2 = _qkv(W * W, d, 194)
    q2 = np.tile(_rng(195).standard_normal(d), (W * W, 1))
    L2 = oracle.num_levels(W // 2)
    pq2 = np.concatenate([np.concatenate([_rng(196 + l).dirichlet(np.ones(2 * 2 ** (l - 1))),
                                          _rng(197 + l).dirichlet(np.ones(2 * 2 ** (l - 1)))])
                          for l in range(1, L2)])
    pk2, pv2 = _pi_2d(W, 2, 198), _pi_2d(W, 2, 199)
    np.testing.assert_allclose(oracle.forward_2d(q2, k2, v2, W, 2, pk2, pv2, piq=pq2),
                               oracle.forward_2d(q2, k2, v2, W, 2, pk2, pv2), rtol=0, atol=1e-12)


def test_linear_rejects_causal_and_rank():
    n, r = 64, 8
    q, k, v = _qkv(n, 4, 200)
    with pytest.raises(RuntimeError):
        oracle.forward_1d(q, k, v, r, _pi_1d(n, r, 1), _pi_1d(n, r, 2), causal=True, piq=_pi_1d(n, r, 3))
    with pytest.raises(RuntimeError):
        oracle.forward_1d(q, k, v, r, _pi_rank_1d(n, r, 2, 1), _pi_rank_1d(n, r, 2, 2), rank=2,
                          piq=_pi_rank_1d(n, r, 2, 3))


# ------------------------------------------------------------------ pin 16
# FMA-linear backward (reading R18): the coarse sources' score gradients flow
# to the coarse queries and through the query coarsening to q and pi^q.
def _grads_torch_linear(q, k, v, r, pk, pv, pq, dout, W=None):
    T = [torch.tensor(x, requires_grad=True) for x in (q, k, v, pk, pv, pq)]
    out = brute.forward_torch(*T[:3], r, T[3], T[4], W=W, piq=T[5])
    (out * torch.tensor(dout)).sum().backward()
    return out.detach().numpy(), [t.grad.numpy() for t in T]


@pytest.mark.parametrize("n,r", [(64, 8), (40, 4), (64, 4)])
def test_linear_backward_matches_autograd_1d(n, r):
    """Oracle FMA-linear gradients (q, k, v, pi^k, pi^v, pi^q) = torch autograd
    of the independent dense formulation, whose forward equals the oracle's."""
    q, k, v = _qkv(n, 6, 201)
    dout = _rng(202).standard_normal((n, 6))
    pk, pv, pq = _pi_1d(n, r, 203), _pi_1d(n, r, 204), _pi_1d(n, r, 205)
    got = oracle.backward_1d(q, k, v, r, pk, pv, dout, piq=pq)
    out, ref = _grads_torch_linear(q, k, v, r, pk, pv, pq, dout)
    np.testing.assert_allclose(out, oracle.forward_1d(q, k, v, r, pk, pv, piq=pq), rtol=0, atol=1e-12)
    assert len(got) == 6
    for g_, r_ in zip(got, ref):
        np.testing.assert_allclose(g_, r_, rtol=0, atol=1e-12)


@pytest.mark.parametrize("W,r", [(8, 2), (12, 2), (8, 1)])
def test_linear_backward_matches_autograd_2d(W, r):
    q, k, v = _qkv(W * W, 6, 206)
    dout = _rng(207).standard_normal((W * W, 6))
    pk, pv, pq = _pi_2d(W, r, 208), _pi_2d(W, r, 209), _pi_2d(W, r, 210)
    got = oracle.backward_2d(q, k, v, W, r, pk, pv, dout, piq=pq)
    out, ref = _grads_torch_linear(q, k, v, r, pk, pv, pq, dout, W=W)
    np.testing.assert_allclose(out, oracle.forward_2d(q, k, v, W, r, pk, pv, piq=pq), rtol=0, atol=1e-12)
    for g_, r_ in zip(got, ref):
        np.testing.assert_allclose(g_, r_, rtol=0, atol=1e-12)


def test_linear_backward_finite_differences():
    """Central differences of the (pinned) FMA-linear forward oracle, every input."""
    n, r, d = 32, 4, 4
    q, k, v = _qkv(n, d, 211)
    dout = _rng(212).standard_normal((n, d))
    pk, pv, pq = _pi_1d(n, r, 213), _pi_1d(n, r, 214), _pi_1d(n, r, 215)
    got = oracle.backward_1d(q, k, v, r, pk, pv, dout, piq=pq)

    def loss(*a):
        return float((dout * oracle.forward_1d(*a[:3], r, a[3], a[4], piq=a[5])).sum())

    g = _rng(216)
    h = 1e-6
    for which in range(6):
        arrs = [q, k, v, pk, pv, pq]
        for flat in g.choice(arrs[which].size, 5, replace=False):
            ix = np.unravel_index(flat, arrs[which].shape)
            plus = [a.copy() for a in arrs]
            minus = [a.copy() for a in arrs]
            plus[which][ix] += h
            minus[which][ix] -= h
            fd = (loss(*plus) - loss(*minus)) / (2 * h)
            assert abs(fd - got[which][ix]) <= 1e-6 * max(1.0, abs(fd)), (which, ix, fd, got[which][ix])


def test_linear_backward_rejects_causal_and_rank():
    n, r = 64, 8
    q, k, v = _qkv(n, 4, 217)
    dout = _rng(218).standard_normal((n, 4))
    with pytest.raises(ValueError):
        oracle.backward_1d(q, k, v, r, _pi_1d(n, r, 1), _pi_1d(n, r, 2), dout, causal=True, piq=_pi_1d(n, r, 3))
    with pytest.raises(ValueError):
        oracle.backward_1d(q, k, v, r, _pi_rank_1d(n, r, 2, 1), _pi_rank_1d(n, r, 2, 2), dout, rank=2,
                           piq=_pi_rank_1d(n, r, 2, 3))


# ------------------------------------------------------------------ pin 17
# Rectangular 2D maps (H rows x W columns, reading R19): the longer side sets
# the depth, a level has ceil(H/s) x ceil(W/s) squares, and the lists are the
# parent's 6 x 6 window minus the 3 x 3 block, clipped per axis.
def _pi_2d_hw(H, W, r, seed, rank=1):
    L = oracle.levels_2d(W, r, H)
    g = _rng(seed)
    parts = [g.standard_normal(2 * r * 2 ** (l - 1)) / np.sqrt(r * 2 ** (l - 1))
             for l in range(1, L) for _ in range(rank)]
    return np.concatenate(parts) if parts else np.zeros(0)


RECT = [(8, 16, 2), (16, 8, 2), (6, 10, 2), (12, 4, 1), (4, 12, 2)]


@pytest.mark.parametrize("H,W,r", RECT)
def test_rect_sets_brute_force_and_closed_form(H, W, r):
    L = oracle.levels_2d(W, r, H)
    nby = W // r
    lists = oracle.lists_2d(W, r, kcap=27, H=H)
    for i in range(H * W):
        x, y = divmod(i, W)
        cell = (x // r) * nby + (y // r)
        near, far = brute.sets_row_2d(W, r, i, H)
        lab = oracle.labels_2d(W, r, i, H)
        assert sorted(np.flatnonzero(lab == 0).tolist()) == near
        covered = list(near)
        for l in range(1, L):
            s = r * 2 ** (l - 1)
            Mx, My = -(-H // s), -(-W // s)
            got = [g for g in lists[cell, l - 1].tolist() if g >= 0]
            assert got == far[l], (H, W, r, i, l)
            qx, qy = (x // r) >> (l - 1), (y // r) >> (l - 1)
            px, py = qx >> 1, qy >> 1
            closed = [u * My + v for u in range(2 * px - 2, 2 * px + 4)
                      for v in range(2 * py - 2, 2 * py + 4)
                      if 0 <= u < Mx and 0 <= v < My and not (abs(u - qx) <= 1 and abs(v - qy) <= 1)]
            assert got == closed
            pix = [xx * W + yy for g in got for xx in range((g // My) * s, min((g // My + 1) * s, H))
                   for yy in range((g % My) * s, min((g % My + 1) * s, W))]
            assert sorted(pix) == sorted(np.flatnonzero(lab == l).tolist())
            covered += pix
        assert sorted(covered) == list(range(H * W))


@pytest.mark.parametrize("H,W,r", RECT)
@pytest.mark.parametrize("p,pl", [(1, False), (2, False), (1, True)])
def test_rect_dense_formulation(H, W, r, p, pl):
    q, k, v = _qkv(H * W, 6, 231)
    pk, pv = _pi_2d_hw(H, W, r, 232, p), _pi_2d_hw(H, W, r, 233, p)
    out = oracle.forward_2d(q, k, v, W, r, pk, pv, rank=p, norm=int(pl), H=H)
    ref = brute.forward_dense_2d(q, k, v, W, r, pk, pv, rank=p, per_level=pl, H=H)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("H,W,r", [(8, 16, 2), (6, 10, 2)])
def test_rect_linear_dense_formulation(H, W, r):
    q, k, v = _qkv(H * W, 6, 234)
    pk, pv, pq = (_pi_2d_hw(H, W, r, 235 + j) for j in range(3))
    out = oracle.forward_2d(q, k, v, W, r, pk, pv, piq=pq, H=H)
    ref = brute.forward_dense_2d(q, k, v, W, r, pk, pv, piq=pq, H=H)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("H,W,r", [(8, 16, 2), (6, 10, 2)])
def test_rect_transpose_equivariance(H, W, r):
    """Transposing an H x W map into a W x H one and swapping pi^(x) with
    pi^(y) transposes the output."""
    d = 6
    q, k, v = _qkv(H * W, d, 241)
    L = oracle.levels_2d(W, r, H)
    pk, pv = _pi_2d_hw(H, W, r, 242), _pi_2d_hw(H, W, r, 243)

    def swap(p):
        out, off = [], 0
        for l in range(1, L):
            s = r * 2 ** (l - 1)
            out += [p[off + s:off + 2 * s], p[off:off + s]]
            off += 2 * s
        return np.concatenate(out)

    T = lambda a, h, w: a.reshape(h, w, d).transpose(1, 0, 2).reshape(h * w, d)   # noqa: E731
    a = oracle.forward_2d(q, k, v, W, r, pk, pv, H=H)
    b = oracle.forward_2d(T(q, H, W), T(k, H, W), T(v, H, W), H, r, swap(pk), swap(pv), H=W)
    np.testing.assert_allclose(T(b, W, H), a, rtol=0, atol=1e-12)


def test_rect_weights_sum_to_one_and_square_case():
    """Joint weights sum to one on a rectangular map (V = 1, pi^v summing to 1
    per axis gives O = 1; whole groups only: the sides are r times powers of
    two), and H = W is the square map."""
    H, W, r = 8, 16, 2
    q, k, _ = _qkv(H * W, 6, 244)
    L = oracle.levels_2d(W, r, H)
    pv = np.concatenate([np.full(2 * r * 2 ** (l - 1), 1.0 / (r * 2 ** (l - 1))) for l in range(1, L)])
    pk = _pi_2d_hw(H, W, r, 245)
    out = oracle.forward_2d(q, k, np.ones((H * W, 6)), W, r, pk, pv, H=H)
    np.testing.assert_allclose(out, 1.0, rtol=0, atol=1e-12)
    W2 = 8
    q2, k2, v2 = _qkv(W2 * W2, 6, 246)
    pk2, pv2 = _pi_2d(W2, 2, 247), _pi_2d(W2, 2, 248)
    np.testing.assert_array_equal(oracle.forward_2d(q2, k2, v2, W2, 2, pk2, pv2, H=W2),
                                  oracle.forward_2d(q2, k2, v2, W2, 2, pk2, pv2))


@pytest.mark.parametrize("H,W,r,lin", [(8, 12, 2, False), (6, 10, 2, True)])
def test_rect_backward_matches_autograd(H, W, r, lin):
    q, k, v = _qkv(H * W, 6, 251)
    dout = _rng(252).standard_normal((H * W, 6))
    pk, pv, pq = (_pi_2d_hw(H, W, r, 253 + j) for j in range(3))
    if lin:
        got = oracle.backward_2d(q, k, v, W, r, pk, pv, dout, piq=pq, H=H)
        T = [torch.tensor(x, requires_grad=True) for x in (q, k, v, pk, pv, pq)]
        out = brute.forward_torch(*T[:3], r, T[3], T[4], W=W, piq=T[5], H=H)
    else:
        got = oracle.backward_2d(q, k, v, W, r, pk, pv, dout, H=H)
        T = [torch.tensor(x, requires_grad=True) for x in (q, k, v, pk, pv)]
        out = brute.forward_torch(*T[:3], r, T[3], T[4], W=W, H=H)
    (out * torch.tensor(dout)).sum().backward()
    for g_, t in zip(got, T):
        np.testing.assert_allclose(g_, t.grad.numpy(), rtol=0, atol=1e-12)
