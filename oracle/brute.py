"""Second, independent formulation of the FMA forward pass (test infrastructure).

TEST INFRASTRUCTURE ONLY.  Pure Python / numpy, float64, for tiny inputs.
It shares no code with ``fma_oracle.c``: index sets are rebuilt here row by
row from the set-builder definitions of Section 3, the coarse keys and values
come from an explicit dense aggregation matrix (Eq. agg1d / Eq. agg2d written
as a matrix product), and the forward pass is a dense masked softmax over the
augmented key set [K; K_bar] (Eq. fma1d / Eq. fma2d read with one joint
normalisation), i.e. an explicit n x (n + R) masked score matrix.  With
coarse level rank p (Sec. 3) the coarse columns are repeated once per basis,
all levels of basis 0 first, where the C oracle orders them by level first.
"""
from __future__ import annotations

import numpy as np


def _levels(ratio: int) -> int:
    L, p = 0, 1
    while p < ratio:
        p, L = 2 * p, L + 1
    return L


# ---------------------------------------------------------------- 1D sets
def sets_row_1d(n: int, r: int, i: int):
    """Near tokens and far groups of query row i, straight from the
    definitions of N(i), F_l(i) and G_l(i).  Returns (near, far) where near is
    a sorted token list and far maps level l to its sorted group indices."""
    L = _levels(n // r)
    near = [j for j in range(n) if abs(j // r - i // r) <= 1]
    used = set(near)
    far = {}
    for l in range(1, L):
        blk = r * 2 ** l
        F = [j for j in range(n) if j not in used and abs(j // blk - i // blk) <= 1]
        s = r * 2 ** (l - 1)
        M = -(-n // s)
        G = [m for m in range(M)
             if all(j in F for j in range(m * s, min((m + 1) * s, n)))]
        far[l] = G
        used.update(F)
    return near, far


def _levels_2d(W: int, r: int, H: int | None) -> int:
    return _levels(max(W if H is None else H, W) // r)


def sets_row_2d(W: int, r: int, i: int, H: int | None = None):
    """2D analogue: near pixels and far squares (index u*My_l + v) of pixel i
    of a map of H rows (default W) and W columns."""
    H = W if H is None else H
    L = _levels_2d(W, r, H)
    xi, yi = divmod(i, W)
    near = [t for t in range(H * W)
            if abs((t // W) // r - xi // r) <= 1 and abs((t % W) // r - yi // r) <= 1]
    used = set(near)
    far = {}
    for l in range(1, L):
        blk = r * 2 ** l
        F = set(t for t in range(H * W) if t not in used
                and abs((t // W) // blk - xi // blk) <= 1
                and abs((t % W) // blk - yi // blk) <= 1)
        s = r * 2 ** (l - 1)
        Mx, My = -(-H // s), -(-W // s)
        G = []
        for u in range(Mx):
            for v in range(My):
                pix = [x * W + y for x in range(u * s, min((u + 1) * s, H))
                       for y in range(v * s, min((v + 1) * s, W))]
                if all(p in F for p in pix):
                    G.append(u * My + v)
        far[l] = G
        used.update(F)
    return near, far


# ------------------------------------------------------ aggregation matrices
def aggregation_matrix_1d(n: int, r: int, pi) -> np.ndarray:
    """Dense [R, n] matrix P with K_bar = P @ K (Eq. agg1d, all levels
    stacked in ascending level order)."""
    pi = np.asarray(pi, dtype=np.float64)
    L = _levels(n // r)
    rows = []
    off = 0
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        p = pi[off:off + s]
        off += s
        for m in range(-(-n // s)):
            row = np.zeros(n)
            for j in range(m * s, min((m + 1) * s, n)):
                row[j] = p[j - m * s]
            rows.append(row)
    return np.array(rows).reshape(-1, n)


def aggregation_matrix_2d(W: int, r: int, pi, H: int | None = None) -> np.ndarray:
    """Dense [R, H*W] matrix with K_bar = P @ K (Eq. agg2d); squares in
    row-major (u, v) order per level; per level pi = [pi_x | pi_y]."""
    H = W if H is None else H
    pi = np.asarray(pi, dtype=np.float64)
    L = _levels_2d(W, r, H)
    rows = []
    off = 0
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        px, py = pi[off:off + s], pi[off + s:off + 2 * s]
        off += 2 * s
        for u in range(-(-H // s)):
            for v in range(-(-W // s)):
                row = np.zeros(H * W)
                for x in range(u * s, min((u + 1) * s, H)):
                    for y in range(v * s, min((v + 1) * s, W)):
                        row[x * W + y] = px[x - u * s] * py[y - v * s]
                rows.append(row)
    return np.array(rows).reshape(-1, H * W)


def rank_bases_1d(n: int, r: int, pi, rank: int):
    """Split rank-p weights (per level: p bases of length s_l, one after the
    other) into p weight vectors in the single-basis layout."""
    pi = np.asarray(pi, dtype=np.float64)
    L = _levels(n // r)
    out = [[] for _ in range(rank)]
    off = 0
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        for b in range(rank):
            out[b].append(pi[off:off + s])
            off += s
    assert off == pi.size, "weight length does not match rank"
    return [np.concatenate(o) if o else np.zeros(0) for o in out]


def rank_bases_2d(W: int, r: int, pi, rank: int, H: int | None = None):
    """2D analogue: per level p consecutive [pi_x | pi_y] pairs."""
    pi = np.asarray(pi, dtype=np.float64)
    L = _levels_2d(W, r, H)
    out = [[] for _ in range(rank)]
    off = 0
    for l in range(1, L):
        s = r * 2 ** (l - 1)
        for b in range(rank):
            out[b].append(pi[off:off + 2 * s])
            off += 2 * s
    assert off == pi.size, "weight length does not match rank"
    return [np.concatenate(o) if o else np.zeros(0) for o in out]


# --------------------------------------------------- dense masked formulation
def mask_1d(n: int, r: int, causal: bool = False) -> np.ndarray:
    """Boolean [n, n + R]: column j < n is fine token j, column n + c is
    coarse row c (levels stacked ascending)."""
    L = _levels(n // r)
    sizes = [r * 2 ** (l - 1) for l in range(1, L)]
    offs = np.cumsum([0] + [-(-n // s) for s in sizes])
    R = int(offs[-1])
    mask = np.zeros((n, n + R), dtype=bool)
    for i in range(n):
        near, far = sets_row_1d(n, r, i)
        for j in near:
            if not causal or j <= i:
                mask[i, j] = True
        for l, G in far.items():
            s = sizes[l - 1]
            for m in G:
                if not causal or min((m + 1) * s, n) - 1 <= i:
                    mask[i, n + offs[l - 1] + m] = True
    return mask


def mask_2d(W: int, r: int, H: int | None = None) -> np.ndarray:
    H = W if H is None else H
    L = _levels_2d(W, r, H)
    sizes = [r * 2 ** (l - 1) for l in range(1, L)]
    offs = np.cumsum([0] + [(-(-H // s)) * (-(-W // s)) for s in sizes])
    n = H * W
    R = int(offs[-1])
    mask = np.zeros((n, n + R), dtype=bool)
    for i in range(n):
        near, far = sets_row_2d(W, r, i, H)
        mask[i, near] = True
        for l, G in far.items():
            for g in G:
                mask[i, n + offs[l - 1] + g] = True
    return mask


def masked_attention(q, kaug, vaug, mask, scale, col_set=None) -> np.ndarray:
    """Row softmax of scale * q kaug^T restricted to mask, times vaug.
    With col_set (one set id per column) the softmax is taken separately over
    the columns of each set and the per-set results are added (a set with no
    visible column adds nothing): the printed per-set normalisation."""
    s = scale * (np.asarray(q, np.float64) @ np.asarray(kaug, np.float64).T)
    s = np.where(mask, s, -np.inf)
    vaug = np.asarray(vaug, np.float64)
    if col_set is None:
        s = s - s.max(axis=1, keepdims=True)
        w = np.exp(s)
        w = w / w.sum(axis=1, keepdims=True)
        return w @ vaug
    col_set = np.asarray(col_set)
    out = np.zeros((s.shape[0], vaug.shape[1]))
    for sid in np.unique(col_set):
        cols = col_set == sid
        ss = s[:, cols]
        vis = np.isfinite(ss).any(axis=1)
        mx = np.where(vis, ss.max(axis=1, initial=-np.inf), 0.0)
        w = np.exp(ss - mx[:, None])
        z = w.sum(axis=1, keepdims=True)
        w = np.where(vis[:, None], w / np.where(z > 0, z, 1.0), 0.0)
        out += w @ vaug[cols]
    return out


def _column_levels(n: int, sizes, counts, rank: int):
    """Set id of every column of [K; K_bar_basis0; K_bar_basis1; ...]: 0 for
    the fine tokens, the level l for a coarse column of level l."""
    lev = np.concatenate([np.full(c, l + 1) for l, c in enumerate(counts)]) if counts else np.zeros(0)
    return np.concatenate([np.zeros(n)] + [lev] * rank)


def forward_dense_1d(q, k, v, r: int, pik=None, piv=None, causal=False, scale=None,
                     rank: int = 1, per_level: bool = False, piq=None):
    """FMA 1D for one (n, d) slice as dense masked attention over [K; K_bar].
    With rank p the augmented set holds one full copy of the coarse columns
    per basis, each copy under the same visibility mask.  per_level: the
    printed normalisation (alpha over the near field, beta^l over all coarse
    columns of level l, every basis included)."""
    n, d = q.shape
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    mask = mask_1d(n, r, causal)
    L = _levels(n // r)
    sizes = [r * 2 ** (l - 1) for l in range(1, L)]
    counts = [-(-n // s) for s in sizes]
    if L > 1:
        bk, bv = rank_bases_1d(n, r, pik, rank), rank_bases_1d(n, r, piv, rank)
        kaug = np.vstack([k] + [aggregation_matrix_1d(n, r, w) @ k for w in bk])
        vaug = np.vstack([v] + [aggregation_matrix_1d(n, r, w) @ v for w in bv])
        mask = np.hstack([mask[:, :n]] + [mask[:, n:]] * rank)
    else:
        kaug, vaug = np.asarray(k, np.float64), np.asarray(v, np.float64)
    col_set = _column_levels(n, sizes, counts, rank) if per_level else None
    if piq is not None and L > 1:
        # FMA-linear: coarse columns scored with the row's own group's coarse query
        qbar = aggregation_matrix_1d(n, r, piq) @ np.asarray(q, np.float64)
        offs = np.cumsum([0] + counts)
        kb = aggregation_matrix_1d(n, r, pik) @ np.asarray(k, np.float64)
        s_far = np.zeros((n, kb.shape[0]))
        for li, sz in enumerate(sizes):
            for c in range(offs[li], offs[li + 1]):
                rows = offs[li] + np.arange(n) // sz
                s_far[:, c] = qbar[rows] @ kb[c]
        s_all = np.hstack([np.asarray(q, np.float64) @ np.asarray(k, np.float64).T, s_far])
        return _masked_softmax_scores(scale * s_all, vaug, mask)
    return masked_attention(q, kaug, vaug, mask, scale, col_set)


def _masked_softmax_scores(s, vaug, mask):
    s = np.where(mask, s, -np.inf)
    s = s - s.max(axis=1, keepdims=True)
    w = np.exp(s)
    return (w / w.sum(axis=1, keepdims=True)) @ np.asarray(vaug, np.float64)


def forward_dense_2d(q, k, v, W: int, r: int, pik=None, piv=None, scale=None, rank: int = 1,
                     per_level: bool = False, piq=None, H: int | None = None):
    H = W if H is None else H
    n, d = q.shape
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    mask = mask_2d(W, r, H)
    L = _levels_2d(W, r, H)
    sizes = [r * 2 ** (l - 1) for l in range(1, L)]
    counts = [(-(-H // s)) * (-(-W // s)) for s in sizes]
    if L > 1:
        bk, bv = rank_bases_2d(W, r, pik, rank, H), rank_bases_2d(W, r, piv, rank, H)
        kaug = np.vstack([k] + [aggregation_matrix_2d(W, r, w, H) @ k for w in bk])
        vaug = np.vstack([v] + [aggregation_matrix_2d(W, r, w, H) @ v for w in bv])
        mask = np.hstack([mask[:, :n]] + [mask[:, n:]] * rank)
    else:
        kaug, vaug = np.asarray(k, np.float64), np.asarray(v, np.float64)
    col_set = _column_levels(n, sizes, counts, rank) if per_level else None
    if piq is not None and L > 1:
        qbar = aggregation_matrix_2d(W, r, piq, H) @ np.asarray(q, np.float64)
        offs = np.cumsum([0] + counts)
        kb = aggregation_matrix_2d(W, r, pik, H) @ np.asarray(k, np.float64)
        s_far = np.zeros((n, kb.shape[0]))
        x, y = np.arange(n) // W, np.arange(n) % W
        for li, sz in enumerate(sizes):
            My = -(-W // sz)
            rows = offs[li] + (x // sz) * My + y // sz
            for c in range(offs[li], offs[li + 1]):
                s_far[:, c] = qbar[rows] @ kb[c]
        s_all = np.hstack([np.asarray(q, np.float64) @ np.asarray(k, np.float64).T, s_far])
        return _masked_softmax_scores(scale * s_all, vaug, mask)
    return masked_attention(q, kaug, vaug, mask, scale, col_set)


def hmatrix_1d(q, k, r: int, pik, piv, causal=False, scale=None) -> np.ndarray:
    """The effective dense n x n attention matrix of the hierarchical
    (H-matrix) view: A[i, j] = alpha_ij on the near field and
    beta_{i,G} * pi^v[j - start(G)] on far groups, so that x_hat = A @ V."""
    n, d = q.shape
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    mask = mask_1d(n, r, causal)
    if _levels(n // r) > 1:
        kaug = np.vstack([k, aggregation_matrix_1d(n, r, pik) @ k])
        P = aggregation_matrix_1d(n, r, piv)
    else:
        kaug, P = np.asarray(k, np.float64), np.zeros((0, n))
    s = scale * (np.asarray(q, np.float64) @ kaug.T)
    s = np.where(mask, s, -np.inf)
    s = s - s.max(axis=1, keepdims=True)
    w = np.exp(s)
    w = w / w.sum(axis=1, keepdims=True)
    return w[:, :n] + w[:, n:] @ P


# ------------------------------------------------ differentiable formulation
def _weight_index_1d(n: int, r: int, rank: int):
    """Per basis b: int [R1, n] index of the weight that multiplies token j in
    coarse row (level, group) -- rows in ascending level, then group -- or -1.
    Indices address the whole rank-p weight vector (per level the p bases one
    after the other)."""
    L = _levels(n // r)
    out = []
    for b in range(rank):
        rows = []
        base = 0
        for l in range(1, L):
            s = r * 2 ** (l - 1)
            for m in range(-(-n // s)):
                row = np.full(n, -1, dtype=np.int64)
                for j in range(m * s, min((m + 1) * s, n)):
                    row[j] = base + b * s + (j - m * s)
                rows.append(row)
            base += rank * s
        out.append(np.array(rows).reshape(-1, n))
    return out


def _weight_index_2d(W: int, r: int, rank: int, H: int | None = None):
    """Per basis: (ix, iy) int [R1, H*W] indices of pi_x[a] and pi_y[b] for
    pixel (x, y) of square (u, v), or -1."""
    H = W if H is None else H
    L = _levels_2d(W, r, H)
    out = []
    for b in range(rank):
        rx, ry = [], []
        base = 0
        for l in range(1, L):
            s = r * 2 ** (l - 1)
            for u in range(-(-H // s)):
                for vv in range(-(-W // s)):
                    ix = np.full(H * W, -1, dtype=np.int64)
                    iy = np.full(H * W, -1, dtype=np.int64)
                    for x in range(u * s, min((u + 1) * s, H)):
                        for y in range(vv * s, min((vv + 1) * s, W)):
                            ix[x * W + y] = base + b * 2 * s + (x - u * s)
                            iy[x * W + y] = base + b * 2 * s + s + (y - vv * s)
                    rx.append(ix)
                    ry.append(iy)
            base += rank * 2 * s
        out.append((np.array(rx).reshape(-1, H * W), np.array(ry).reshape(-1, H * W)))
    return out


def forward_torch(q, k, v, r: int, pik, piv, causal=False, scale=None, rank: int = 1, per_level=False,
                  W: int | None = None, piq=None, H: int | None = None):
    """Differentiable fp64 torch version of the dense masked formulation (1D,
    or 2D when W is given): the aggregation matrices are built from the
    weight tensors by indexing, so autograd yields d/dq, d/dk, d/dv and
    d/dpi.  Inputs are torch float64 tensors (requires_grad as needed).
    piq (FMA-linear, rank 1, joint): every coarse column is scored with the
    row's own group's coarse query at that column's level."""
    import torch
    n, d = q.shape
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    two_d = W is not None
    if two_d and H is None:
        H = W
    mask = mask_2d(W, r, H) if two_d else mask_1d(n, r, causal)
    L = _levels_2d(W, r, H) if two_d else _levels(n // r)
    cols_k, cols_v = [k], [v]
    col_set = None
    qbar = None
    if L > 1:
        if two_d:
            for ix, iy in _weight_index_2d(W, r, rank, H):
                tx, ty = torch.from_numpy(ix), torch.from_numpy(iy)
                on = tx >= 0
                ak = torch.where(on, pik[tx.clamp(min=0)] * pik[ty.clamp(min=0)], torch.zeros((), dtype=q.dtype))
                av = torch.where(on, piv[tx.clamp(min=0)] * piv[ty.clamp(min=0)], torch.zeros((), dtype=q.dtype))
                cols_k.append(ak @ k)
                cols_v.append(av @ v)
                if piq is not None:
                    aq = torch.where(on, piq[tx.clamp(min=0)] * piq[ty.clamp(min=0)], torch.zeros((), dtype=q.dtype))
                    qbar = aq @ q
            sizes = [r * 2 ** (l - 1) for l in range(1, L)]
            counts = [(-(-H // s)) * (-(-W // s)) for s in sizes]
        else:
            for idx in _weight_index_1d(n, r, rank):
                t = torch.from_numpy(idx)
                on = t >= 0
                cols_k.append(torch.where(on, pik[t.clamp(min=0)], torch.zeros((), dtype=q.dtype)) @ k)
                cols_v.append(torch.where(on, piv[t.clamp(min=0)], torch.zeros((), dtype=q.dtype)) @ v)
                if piq is not None:
                    qbar = torch.where(on, piq[t.clamp(min=0)], torch.zeros((), dtype=q.dtype)) @ q
            sizes = [r * 2 ** (l - 1) for l in range(1, L)]
            counts = [-(-n // s) for s in sizes]
        mask = np.hstack([mask[:, :n]] + [mask[:, n:]] * rank)
        if per_level:
            col_set = _column_levels(n, sizes, counts, rank)
    kaug, vaug = torch.cat(cols_k, 0), torch.cat(cols_v, 0)
    s = scale * (q @ kaug.T)
    if qbar is not None:
        # column c of level l (coarse rows offs[l] ..) is scored by row i with
        # the coarse query of i's own level-l group
        kb = torch.cat(cols_k[1:], 0)
        offs = np.cumsum([0] + counts)
        sel = np.zeros((n, kb.shape[0]), dtype=np.int64)
        tok = np.arange(n)
        for li, sz in enumerate(sizes):
            if two_d:
                M = -(-W // sz)
                rows = offs[li] + (tok // W // sz) * M + (tok % W) // sz
            else:
                rows = offs[li] + tok // sz
            sel[:, offs[li]:offs[li + 1]] = rows[:, None]
        ti = torch.from_numpy(sel)
        s_far = (qbar[ti] * kb[None, :, :]).sum(-1)
        s = torch.cat([s[:, :n], scale * s_far], 1)
    m = torch.from_numpy(mask)
    s = s.masked_fill(~m, float("-inf"))
    if col_set is None:
        return torch.softmax(s, dim=1) @ vaug
    out = torch.zeros_like(q)
    for sid in np.unique(col_set):
        cols = torch.from_numpy(col_set == sid)
        ss = s[:, cols]
        vis = torch.isfinite(ss).any(dim=1, keepdim=True)
        w = torch.softmax(torch.where(vis, ss, torch.zeros((), dtype=q.dtype)), dim=1)
        w = torch.where(vis & torch.isfinite(ss), w, torch.zeros((), dtype=q.dtype))
        w = w / torch.where(vis, w.sum(dim=1, keepdim=True), torch.ones((), dtype=q.dtype))
        out = out + w @ vaug[cols]
    return out
