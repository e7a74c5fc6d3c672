"""Host-side emulation of the address arithmetic of the library's kernels
(test infrastructure; no device access).

Driven by the library's own plan (paper_2310_11960_amd.fma_plan_params), it
restates, statement by statement, how the kernels form every global address,
LDS destination, ring slot and staged output row, and checks them against the
buffers' sizes and against what the data layout says they must be:

  attend_mfma_kernel / attend_kernel tile stream (attend_mfma.hip):
    - the persistent schedule visits every query block exactly once, for any
      grid size;
    - Q, near and coarse tiles: every 16-byte load of every lane stays inside
      its slice of its tensor, the eight rows a load covers are the eight
      consecutive tokens the lane offsets assume (the load's base is taken
      from one lane: it must be the same for all lanes), the near tiles cover
      exactly the near field, and every interaction-list slot maps to a row
      of its own coarse set (or is empty);
  coarsen1d_stream / coarsen2d_stream (coarsen.hip):
    - every step's rows and weight gathers stay inside their tensors and
      weight vectors;
    - the groups (squares) that close at a step are a prefix of the sets,
      the same ones that close by division, and the closed group index is
      the right one;
    - at most 16 closed rows are ever staged, every staged row and every
      partial-sum row lies inside the workspace.

A failed check raises AssertionError with the offending values.
"""
from __future__ import annotations

import numpy as np

KT = 64        # keys per tile
ROWB = 128     # bytes per bf16 row of 64 channels
MAX_SLOTS = 448
MAX_PAIR_SLOTS = 768   # the paired 2D kernel: both cells' tables side by side
K1D, K2D = 3, 27


# ----------------------------------------------------------------- closed-form lists
def list1d_entry(b, l, j, M, causal):
    """Vectorised over b (numpy int array): the fused kernel's closed form."""
    q = b >> (l - 1)
    p = q >> 1
    even = (q & 1) == 0
    if j == 0:
        g = 2 * p - 2
    elif j == 1:
        g = np.where(even, 2 * p + 2, 2 * p - 1)
    else:
        g = 2 * p + 3
    bad = (g < 0) | (g >= M)
    if causal:
        bad |= g > q - 2
    return np.where(bad, -1, g)


def window_slot(j, ox, oy):
    """Vectorised over ox, oy (arrays); j scalar."""
    au = np.empty_like(ox)
    av = np.empty_like(ox)
    top = j < 6 * ox
    au[top] = j // 6
    av[top] = j - 6 * (j // 6)
    mid = (~top) & (j < 6 * ox + 9)
    t = j - 6 * ox
    k = t % 3
    au[mid] = (ox + t // 3)[mid]
    av[mid] = np.where(k < oy, k, k + 3)[mid]
    bot = ~(top | mid)
    t2 = j - 6 * ox - 9
    au[bot] = (ox + 3 + t2 // 6)[bot]
    av[bot] = (t2 % 6)[bot]
    return au, av


def list2d_entry(cx, cy, l, j, M, My):
    qx, qy = cx >> (l - 1), cy >> (l - 1)
    au, av = window_slot(j, 1 + (qx & 1), 1 + (qy & 1))
    u = 2 * (qx >> 1) - 2 + au
    v = 2 * (qy >> 1) - 2 + av
    bad = (u < 0) | (u >= M) | (v < 0) | (v >= My)
    return np.where(bad, -1, u * My + v)


def list2d_slot_of(qx, qy, u, v):
    """The backward reduction's inverse of list2d_entry (bwd_reduce): the
    entry j of level group (qx, qy)'s list that names square (u, v), or -1."""
    au, av = u - (2 * (qx >> 1) - 2), v - (2 * (qy >> 1) - 2)
    if au < 0 or au >= 6 or av < 0 or av >= 6:
        return -1
    ox, oy = 1 + (qx & 1), 1 + (qy & 1)
    if au < ox:
        return au * 6 + av
    if au < ox + 3:
        if oy <= av < oy + 3:
            return -1
        return 6 * ox + (au - ox) * 3 + (av if av < oy else av - 3)
    return 6 * ox + 9 + (au - ox - 3) * 6 + av


# ----------------------------------------------------------------- fused attention
def near_in_order(lo, nb, k):
    """The k-th of nb (1 .. 3) consecutive near blocks (2D: rows / columns of
    near cells) starting at lo, in ascending order of index mod 3 (the tile
    walk's near-field order); vectorised over lo and nb."""
    lo = np.asarray(lo)
    nb = np.asarray(nb)
    three = lo + (k - lo % 3 + 3) % 3
    two = np.where(lo % 3 == 2, lo + 1 - k, lo + k)
    return np.where(nb == 3, three, np.where(nb == 2, two, lo))


def schedule_blocks(total, G):
    """The persistent schedule of attend_mfma_kernel: workgroup x takes
    blocks blk_first, blk_first + gx, ... < blk_end.  Returns the list of
    each workgroup's blocks."""
    nx = G if G < 8 else 8
    out = []
    for bx in range(G):
        xg, jg = bx % nx, bx // nx
        gx = (G - 1 - xg) // nx + 1
        blk_end = total * (xg + 1) // nx
        blk_first = total * xg // nx + jg
        out.append(range(blk_first, blk_end, gx))
    return out


def check_schedule(total, grids):
    for G in grids:
        G = min(G, total) if total > 0 else G
        if total == 0:
            continue
        seen = np.zeros(total, dtype=np.int64)
        for r in schedule_blocks(total, G):
            if len(r):
                seen[np.asarray(r)] += 1
        assert (seen == 1).all(), ("schedule", total, G, int((seen != 1).sum()))


def _coarse_rows(P, geom, blocks_qt):
    """Interaction-list slot table (FMA_SLOT_ENTRY) for the query blocks
    blocks_qt: int array [nblk, nslot] of coarse rows (-1 empty)."""
    nslot, sgrp, rank = P["nslot"], P["slot_group"], P["rank"]
    K = K2D if geom == "2d" else K1D
    sets = P["sets"]
    out = np.full((len(blocks_qt), max(nslot, 1)), -1, dtype=np.int64)
    for e in range(nslot):
        if P["norm_level"]:
            lev, rem = divmod(e, sgrp)
            b, j = divmod(rem, K)
            st = lev * rank + b
            if b >= rank:
                continue
        else:
            st, j = divmod(e, K)
        assert 0 <= st < len(sets), ("slot set", e, st)
        M, My, lvl, off = sets[st]["M"], sets[st]["My"], sets[st]["lvl"], sets[st]["off"]
        if geom == "2d":
            cx, cy = blocks_qt // P["nby"], blocks_qt % P["nby"]
            gi = list2d_entry(cx, cy, lvl, j, M, My)
            nrows = M * My
        else:
            gi = list1d_entry(blocks_qt, lvl, j, M, P["causal"])
            nrows = M
        assert (gi < nrows).all()
        out[:, e] = np.where(gi >= 0, off + gi, -1)
        # a set's rows are its own block of the coarse arrays
        ok = gi < 0
        ok |= (off + gi >= off) & (off + gi < off + nrows) & (off + gi < P["R"])
        assert ok.all(), ("coarse row outside its set", e, st)
    return out


def check_attend_issue(P, geom, dense=False, grids=(1, 3, 8, 9, 100, 1024, 2048, 4096, 8192), near_order="ascending"):
    """The tile stream of attend_mfma_kernel (FMA_ISSUE_SCALAR in 1D,
    FMA_ISSUE_VGPR in 2D and for the dense reference) for every query block.
    near_order: "ascending" (the kernel's order: near blocks, 2D cells
    row-major, in ascending position); "mod3" walks them in ascending index
    mod 3 (an alternative order, measured and not used; 1D causal and dense
    stay ascending)."""
    n, r, qtile = P["n"], P["block"], P["qtile"]
    nslice, R, side, nbx, nby, H = P["nslice"], P["R"], P["side"], P["nbx"], P["nby"], P["height"]
    causal = P["causal"]
    if dense:
        qtile = 128 if n % 128 == 0 else 64
        tps = n // qtile
        nslot = 0
    else:
        tps = P["tiles_per_slice"]
        nslot = P["nslot"]
    NW = qtile // 32
    assert qtile % 32 == 0 and NW in (2, 4, 6, 8), ("workgroup shape", qtile)
    nq = (NW + 3) // 4
    nctile = (nslot + KT - 1) // KT
    assert nslot <= MAX_SLOTS
    total = tps * nslice
    check_schedule(total, grids)
    if total == 0:
        return 0
    qt = np.arange(tps, dtype=np.int64)
    lg_r = r.bit_length() - 1
    tpc = (r * r) // KT if geom == "2d" else 1
    if geom == "2d":
        assert (r * r) % KT == 0, "2D cell must be whole tiles"
        assert 1 << lg_r == r

    def block_token(p):
        if geom == "2d":
            cx, cy = qt // nby, qt % nby
            return (cx * r + (p >> lg_r)) * side + cy * r + (p & (r - 1))
        return qt * qtile + p

    nloads = 0
    # Q tiles: 128 query rows per tile, 8 per load
    for ilt in range(nq):
        for j in range(16):
            i, half = j & 7, j >> 3
            p0 = ilt * 128 + half * 64 + 8 * i
            if p0 >= qtile:
                p0 -= qtile * (p0 // qtile)
            base = block_token(p0)
            for lr in range(8):
                assert (block_token(p0 + lr) == base + lr).all(), ("Q rows not contiguous", ilt, j, lr)
            assert (base >= 0).all() and (base + 8 <= n).all(), ("Q load outside the slice", ilt, j)
            nloads += len(base)
    # near tiles
    if geom == "2d":
        cx, cy = qt // nby, qt % nby
        dx0 = np.where(cx > 0, -1, 0)
        dx1 = np.where(cx + 1 < nbx, 1, 0)
        dy0 = np.where(cy > 0, -1, 0)
        dy1 = np.where(cy + 1 < nby, 1, 0)
        ncy = dy1 - dy0 + 1
        nnear = (dx1 - dx0 + 1) * ncy * tpc
        covered = {}
        sample = set(range(min(tps, 48))) | set(range(max(tps - 48, 0), tps)) | set(range(0, tps, max(tps // 32, 1)))
        ncx = dx1 - dx0 + 1
        for t in range(int(nnear.max())):
            act = t < nnear
            ci, sub = t // tpc, t % tpc
            if near_order == "mod3":
                ux = near_in_order(cx + dx0, ncx, ci // ncy)
                uy = near_in_order(cy + dy0, ncy, ci % ncy)
            else:
                ux = cx + dx0 + ci // ncy
                uy = cy + dy0 + ci % ncy
            assert ((ux >= 0) & (ux < nbx) & (uy >= 0) & (uy < nby))[act].all(), ("near cell off the map", t)
            for i in range(8):
                p0 = sub * KT + 8 * i
                tok = (ux * r + (p0 >> lg_r)) * side + uy * r + (p0 & (r - 1))
                for lr in range(8):
                    p = p0 + lr
                    t2 = (ux * r + (p >> lg_r)) * side + uy * r + (p & (r - 1))
                    assert (t2 == tok + lr)[act].all(), ("near rows not contiguous", t, i, lr)
                assert ((tok >= 0) & (tok + 8 <= n))[act].all()
                nloads += 2 * int(act.sum())
                for b in sample:   # coverage on a sample of blocks (first, last, spread)
                    if act[b]:
                        covered.setdefault(b, set()).update(range(int(tok[b]), int(tok[b]) + 8))
        for b, toks in covered.items():
            x0, y0 = (b // nby) * r, (b % nby) * r
            want = {x * side + y for x in range(max(x0 - r, 0), min(x0 + 2 * r, H))
                    for y in range(max(y0 - r, 0), min(y0 + 2 * r, side))}
            assert toks == want, ("2D near field", b)
    else:
        if dense:
            klo = np.zeros_like(qt)
            hi = np.minimum((qt + 1) * qtile, n) if causal else np.full_like(qt, n)
            nnear = (hi + KT - 1) // KT
        else:
            klo = np.where(qt > 0, (qt - 1) * r, 0)
            hi = np.minimum((qt + 1) * r if causal else (qt + 2) * r, n)
            assert ((hi - klo) % KT == 0).all(), "near field not whole tiles"
            nnear = (hi - klo) // KT
        ordered = near_order == "mod3" and not dense and not causal
        seen = np.zeros((len(qt), int(nnear.max())), dtype=np.int64)
        for t in range(int(nnear.max())):
            act = t < nnear
            if ordered:
                tpb = r >> 6
                k, sub = divmod(t, tpb)
                lo = np.maximum(qt - 1, 0)
                nbk = np.minimum(qt + 1, nbx - 1) - lo + 1
                tok0 = near_in_order(lo, nbk, k) * r + sub * KT
            else:
                tok0 = klo + t * KT
            seen[:, t] = np.where(act, tok0, -1)
            for i in range(8):
                tok = tok0 + 8 * i
                assert ((tok >= 0) & (tok + 8 <= n))[act].all(), ("near load outside the slice", t, i)
                nloads += 2 * int(act.sum())
        if not dense:
            # the near tiles are exactly N(i) of the block (causal: up to the block's end), each once
            lo_want = np.maximum(qt - 1, 0) * r
            assert (klo == lo_want).all() and (klo + nnear * KT == hi).all()
            want = klo[:, None] + KT * np.arange(seen.shape[1])[None, :]
            want = np.where(np.arange(seen.shape[1])[None, :] < nnear[:, None], want, -1)
            assert (np.sort(seen, 1) == np.sort(want, 1)).all(), "near tiles do not cover the near field once"
            if not causal and r % KT == 0 and nbx >= 3:
                # interior blocks read each near block in the same step: step of block x = x mod 3
                tpb = r >> 6
                inner = (qt >= 1) & (qt + 1 < nbx)
                for t in range(3 * tpb):
                    x = seen[inner, t] // r
                    if ordered:
                        assert (x % 3 == t // tpb).all(), "near order"
    # coarse tiles
    if nctile:
        rows = _coarse_rows(P, geom, qt)
        for ct in range(nctile):
            for i in range(8):
                for lrow in range(8):
                    e = ct * KT + 8 * i + lrow
                    row = rows[:, e] if e < nslot else np.full(len(qt), -1)
                    row = np.maximum(row, 0)
                    assert ((row >= 0) & (row < R)).all(), ("coarse row outside the slice", ct, i, lrow)
            nloads += 16 * len(qt)
    # LDS: a load's 64 lanes write 1 KB at row 8i of an 8 KB half-stage
    for i in range(8):
        assert i * 1024 + 64 * 16 <= 8 * 1024
    return nloads * nslice


# ----------------------------------------------------------------- coarsening
def _stream_weight_loads(sets):
    for lim, w in ((4, 1), (8, 2), (12, 3), (16, 4), (24, 6), (32, 8)):
        if sets <= lim:
            return w
    return 0


def _stream2d_cols(s):
    return 32 // s if s <= 32 else 1


def _stream2d_weight_loads(sets):
    for lim, w in ((4, 1), (8, 2), (16, 4), (32, 8)):
        if sets <= lim:
            return w
    return 0


def coarsening_passes(P):
    """The passes launch_coarsen makes: (first set, count) pairs."""
    sets, nsets = P["sets"], P["nsets"]
    stream = P["dtype"] == 1 and P["depth"] > 0
    out, v0 = [], 0
    while v0 < nsets:
        if stream and P["ndim"] == 2:
            cols, cnt = 0, 0
            while v0 + cnt < nsets and cols + _stream2d_cols(sets[v0 + cnt]["size"]) <= 32:
                cols += _stream2d_cols(sets[v0 + cnt]["size"])
                cnt += 1
        else:
            cnt = min(nsets - v0, 32 if stream else 16)
        assert cnt > 0, "empty coarsening pass"
        out.append((v0, cnt))
        v0 += cnt
    return out


def check_coarsen1d_stream(P):
    """coarsen1d_stream, every pass and every unit: rows, weight gathers,
    closing prefix, staging and output rows."""
    n, nslice, R = P["n"], P["nslice"], P["R"]
    CW, upz, D = P["chunk"], P["nchunk"], P["depth"]
    heads, w_stride, wlen, heads_w = P["heads"], P["w_stride"], P["wlen"], P["heads_w"]
    assert CW % 16 == 0 and n % 16 == 0
    nsteps = CW >> 4
    U = 2 * nslice * upz
    assert upz == -(-n // CW)
    max_staged = 0
    for v0, cnt in coarsening_passes(P):
        ps = P["sets"][v0:v0 + cnt]
        nlev = cnt
        NWD = _stream_weight_loads(nlev)
        assert NWD and nlev <= 4 * NWD
        need = D * (2048 + 256 * NWD) + 64 + 2048 + 64
        assert need <= P["wave_lds"] and 4 * P["wave_lds"] <= P["coarsen_smem"], ("LDS", need, P["wave_lds"])
        first_partial = P["first_partial"] - v0
        CG = 2 if NWD > 4 else 1
        ndir = 0
        while ndir < nlev and ps[ndir]["size"] <= CW:
            ndir += 1
        for l in range(nlev):
            assert ps[l]["size"] % 16 == 0 and (l == 0 or ps[l]["size"] >= ps[l - 1]["size"])
        first16 = ps[0]["size"] >> 4 if ndir > 0 else 1 << 30
        lvl0 = ps[0]["lvl"]
        cwsh = 0
        while ndir > 0 and (ps[0]["size"] << cwsh) < CW:
            cwsh += 1
        if ndir > 0:
            assert ps[0]["size"] << cwsh == CW
        # weights: per load i, lane L gathers weight L % 16 of set 4 i + L / 16
        wsz, wof, wmask = [], [], []
        for i in range(NWD):
            for lane in range(64):
                lv = 4 * i + (lane >> 4)
                s, o = 16, 0
                if lv < nlev:
                    s, o = ps[lv]["size"], ps[lv]["woff"] + (lane & 15)
                wsz.append(s)
                wof.append(o)
                wmask.append(s // CW - 1 if s > CW else 0)
        wsz, wof, wmask = np.array(wsz), np.array(wof), np.array(wmask)
        assert ((wsz % CW == 0) | (wsz <= CW)).all()
        for c in range(upz):
            t0 = c * CW
            inv = min((n - t0) >> 4, nsteps)
            assert t0 + 16 * inv <= n and inv >= 1
            # weight gathers over the unit's steps
            ipos = (c & wmask) * CW
            for _ in range(inv):
                idx = wof + ipos
                assert ((idx >= 0) & (idx < max(wlen, 1))).all(), ("weight index", c)
                ipos = ipos + 16
                ipos = np.where(ipos >= wsz, ipos - wsz, ipos)
            # closing and staging
            nout, left0, kk = 0, first16, 0
            for st in range(nsteps):
                left0 -= 1
                if left0 > 0:
                    continue
                left0 = first16
                kk += 1
                rel = 16 * (st + 1)
                lc = 0
                while lc < ndir and not (kk & ((1 << (ps[lc]["lvl"] - lvl0)) - 1)):
                    lc += 1
                ref = [l for l in range(ndir) if rel % ps[l]["size"] == 0]
                assert ref == list(range(lc)), ("closing prefix", c, st, ref, lc)
                for g in range(CG):
                    cn = min(lc - 16 * g, 16)
                    if cn <= 0:
                        break
                    if nout + cn > 16:
                        nout = 0
                    for lv in range(cn):
                        l = 16 * g + lv
                        se = ps[l]["lvl"] - lvl0
                        m = (c << (cwsh - se)) + (kk >> se) - 1
                        assert m == (t0 + rel) // ps[l]["size"] - 1, ("closed group", c, st, l)
                        slot = nout + lv
                        assert 0 <= slot < 16
                        if m < ps[l]["M"]:
                            for zs in (0, 2 * nslice - 1):
                                row = zs * R + ps[l]["off"] + m
                                assert 0 <= row < 2 * nslice * R
                    nout += cn
                    max_staged = max(max_staged, nout)
            # partial rows of the sets wider than the unit
            for l in range(ndir, nlev):
                gi = l - first_partial
                assert 0 <= gi < P["npartial"], ("partial set", l, gi)
                for zs in (0, 2 * nslice - 1):
                    idx = (zs * P["npartial"] + gi) * P["part_count"] + c
                    assert 0 <= idx < 2 * nslice * P["npartial"] * P["part_count"]
        # each head's weights lie inside the weight buffer
        for sl in (0, nslice - 1):
            if nslice:
                assert (sl % heads) * w_stride + wlen <= heads_w * wlen
        assert U >= 0
    assert max_staged <= 16
    return max_staged


def check_coarsen2d_stream(P):
    """coarsen2d_stream, every pass and tile: pixel rows, x and y weight
    gathers, closing prefix, staging, output squares and partial rows."""
    W, H, nslice, R = P["side"], P["height"], P["nslice"], P["R"]
    D, ntx, nty = P["depth"], P["tiles_x"], P["tiles_y"]
    wlen = P["wlen"]
    assert W % 32 == 0 and H % 32 == 0 and nty == W // 32 and ntx == H // 32 and P["nchunk"] == ntx * nty
    max_staged = 0
    for v0, cnt in coarsening_passes(P):
        ps = P["sets"][v0:v0 + cnt]
        nlev = cnt
        ncols = sum(_stream2d_cols(e["size"]) for e in ps)
        ndir = max([e + 1 for e in range(nlev) if ps[e]["size"] <= 32], default=0)
        NWY = _stream2d_weight_loads(nlev)
        CG = 2 if ncols > 16 else 1
        assert NWY and nlev <= 4 * NWY and ncols <= 16 * CG
        need = D * (2048 + 256 * NWY + 256) + 64 + 2048 + 64
        assert need <= P["wave_lds"] and 4 * P["wave_lds"] <= P["coarsen_smem"], ("LDS", need)
        assert nlev <= 64
        first_partial = P["first_partial"] - v0
        # the lane's (set, square column) per accumulator column
        colmap = []
        for e in range(nlev):
            for j in range(_stream2d_cols(ps[e]["size"])):
                colmap.append((e, j))
        for tx in range(ntx):
            for ty in range(nty):
                # rows streamed: 32 rows of 32 pixels, two 16-pixel halves each
                assert 32 * tx + 32 <= H and 32 * ty + 32 <= W
                for e in range(nlev):
                    s, wo = ps[e]["size"], ps[e]["woff"]
                    for y in range(16):
                        yo0 = wo + s + (y & (s - 1)) if s <= 32 else wo + s + ((32 * ty) & (s - 1)) + y
                        yo1 = wo + s + ((16 + y) & (s - 1)) if s <= 32 else wo + s + ((32 * ty) & (s - 1)) + 16 + y
                        assert wo + s <= yo0 < wo + 2 * s and wo + s <= yo1 < wo + 2 * s and yo1 < wlen
                    ixb = wo if s <= 32 else wo + ((32 * tx) & (s - 1))
                    ixm = s - 1 if s <= 32 else 31
                    for x in range(32):
                        assert wo <= ixb + (x & ixm) < wo + s
                nout = 0
                for x in range(32):
                    lc = lcc = 0
                    while lc < ndir and not ((x + 1) & (ps[lc]["size"] - 1)):
                        lcc += _stream2d_cols(ps[lc]["size"])
                        lc += 1
                    ref = [e for e in range(ndir) if (x + 1) % ps[e]["size"] == 0]
                    assert ref == list(range(lc)), ("closing prefix 2D", tx, ty, x)
                    for g in range(CG):
                        cn = min(lcc - 16 * g, 16)
                        if cn <= 0:
                            break
                        if nout + cn > 16:
                            nout = 0
                        for lv in range(cn):
                            e, cj = colmap[16 * g + lv]
                            s, M, My = ps[e]["size"], ps[e]["M"], ps[e]["My"]
                            ssh = s.bit_length() - 1
                            u = (32 * tx + x) >> ssh
                            v = ((32 * ty) >> ssh) + cj
                            assert u == (32 * tx + x) // s and v == (32 * ty + cj * s) // s
                            assert u < M and v < My, ("whole tiles close only in-map squares", u, v)
                            if u < M and v < My:
                                for zs in (0, 2 * nslice - 1):
                                    row = zs * R + ps[e]["off"] + u * My + v
                                    assert 0 <= row < 2 * nslice * R
                        nout += cn
                        max_staged = max(max_staged, nout)
                for e in range(ndir, nlev):
                    gi = e - first_partial
                    assert 0 <= gi < P["npartial"], ("partial set 2D", e, gi)
                    t = tx * nty + ty
                    for zs in (0, 2 * nslice - 1):
                        idx = (zs * P["npartial"] + gi) * P["part_count"] + t
                        assert 0 <= idx < 2 * nslice * P["npartial"] * P["part_count"]
    assert max_staged <= 16
    return max_staged


def check_pair_issue(P, grids=(1, 3, 8, 9, 100, 1024, 2048, 4096, 8192)):
    """The 2D tile stream with cells taken in horizontal pairs (GEOM_2DP):
    two cells (x, 2c) and (x, 2c + 1) per workgroup, one Q tile of their 128
    queries, the union of their near fields walked column by column (shared
    columns first, then the left cell's, then the right cell's), then each
    cell's coarse tiles from its own half of the slot table."""
    n, r, side, nbx, nby, R, nslice = P["n"], P["block"], P["side"], P["nbx"], P["nby"], P["R"], P["nslice"]
    nslot = P["nslot"]
    assert r == 8 and nby % 2 == 0 and P["tiles_per_slice"] == nbx * nby
    nctile = (nslot + KT - 1) // KT
    assert nslot <= MAX_SLOTS and 2 * nctile * KT <= MAX_PAIR_SLOTS, "both cells' tables must fit the slot table"
    tps = P["tiles_per_slice"] // 2
    check_schedule(tps * nslice, grids)
    qt = np.arange(tps, dtype=np.int64)
    half = nby // 2
    cx, cy = qt // half, 2 * (qt % half)
    # Q tile: 128 rows, 8 per load, left cell then right cell
    def tok_of(p):
        c, q = p >> 6, p & 63
        return (cx * r + (q >> 3)) * side + (cy + c) * r + (q & 7)
    nloads = 0
    for j in range(16):
        i, hf = j & 7, j >> 3
        p0 = hf * 64 + 8 * i
        base = tok_of(p0)
        for lr in range(8):
            assert (tok_of(p0 + lr) == base + lr).all(), ("pair Q rows", j, lr)
        assert ((base >= 0) & (base + 8 <= n)).all()
        nloads += len(qt)
    # near window
    dx0 = np.where(cx > 0, -1, 0)
    dx1 = np.where(cx + 1 < nbx, 1, 0)
    ncx = dx1 - dx0 + 1
    nA = np.where(cy > 0, 1, 0)
    nB = np.where(cy + 2 < nby, 1, 0)
    ncy = 2 + nA + nB
    nnear = ncx * ncy
    cells = {0: [set() for _ in qt], 1: [set() for _ in qt]}
    for t in range(int(nnear.max())):
        act = t < nnear
        cs, row = t // ncx, t % ncx
        ux = cx + dx0 + row
        uy = np.where(cs < 2, cy + cs, np.where((cs == 2) & (nA == 1), cy - 1, cy + 2))
        grp = np.where(uy <= cy + 1, 1, 0) | np.where(uy >= cy, 2, 0)
        assert ((ux >= 0) & (ux < nbx) & (uy >= 0) & (uy < nby))[act].all(), ("pair near cell off the map", t)
        if t == 0:
            assert (grp == 3).all(), "the first near tile must be shared (FIRST path)"
        for i in range(8):
            tok = (ux * r + i) * side + uy * r
            assert ((tok >= 0) & (tok + 8 <= n))[act].all()
            nloads += 2 * int(act.sum())
        for b in np.nonzero(act)[0]:
            for c in (0, 1):
                if (grp[b] >> c) & 1:
                    cells[c][b].add((int(ux[b]), int(uy[b])))
    for b in range(len(qt)):
        for c in (0, 1):
            x0, y0 = int(cx[b]), int(cy[b]) + c
            want = {(x, y) for x in range(x0 - 1, x0 + 2) for y in range(y0 - 1, y0 + 2) if 0 <= x < nbx and 0 <= y < nby}
            assert cells[c][b] == want, ("pair near field", b, c)
    # coarse tiles: each cell's table (joint or per-level slot layout,
    # FMA_SLOT_ENTRY) in its half; empty slots read row 0
    for c in (0, 1):
        rows = _coarse_rows(P, "2d", cx * nby + cy + c)
        assert ((np.where(rows >= 0, rows, 0) >= 0) & (rows < R)).all()
        assert c * nctile * KT + nslot <= MAX_PAIR_SLOTS
        nloads += 16 * nctile * len(qt)
    return nloads * nslice


def small_blocks(P):
    """Blocks smaller than a wave (1D r < 64, 2D cells below 8 x 8), and any
    head dim but 64: both dtypes take the register-staged kernel
    (attend_kernel, row_source)."""
    return P["block"] < (64 if P["ndim"] == 1 else 8) or P["head_dim"] != 64


def check_generic_issue(P):
    """The rows attend_kernel loads (row_source) for every query block of a
    plan of small blocks: the near field's tokens packed 64 to a tile (1D:
    klo .. khi; 2D: the in-map 3 x 3 cells, cell after cell), rows past it
    empty; then the coarse slots.  Every token lies in the slice and the
    near tiles cover exactly the near field, once.  The lanes past the
    block (qtile < 32) repeat query ql mod qtile, inside the block."""
    n, r, nbx, nby, side, R = P["n"], P["block"], P["nbx"], P["nby"], P["side"], P["R"]
    causal, qtile, tps, d = P["causal"], P["qtile"], P["tiles_per_slice"], P["head_dim"]
    assert 0 < qtile <= 256 and (qtile <= 32 or qtile % 32 == 0) and (P["ndim"] == 2 or qtile == r)
    assert d in (32, 64, 128)
    NW = (qtile + 31) // 32
    assert NW in (1, 2, 4, 6, 8), ("workgroup shape", qtile)
    qt = np.arange(tps, dtype=np.int64)
    nloads = 0
    for lane in range(32 * NW):   # lanes past a block smaller than a wave repeat a query
        ql = lane if lane < qtile else lane % qtile
        if P["ndim"] == 2:
            cx, cy = qt // nby, qt % nby
            tok = (cx * r + ql // r) * side + cy * r + ql % r
        else:
            tok = qt * qtile + ql
        assert ((tok >= 0) & (tok < n)).all(), ("query row outside the slice", lane)
    # the tile loads: 64 rows of d channels in 16-byte chunks, every chunk of
    # every row loaded once (K: KCHUNKS chunks; V: bf16 key pairs, fp32 rows)
    esize = 2 if P["dtype"] == 1 else 4
    kcols = d * esize // 16
    kchunks = 64 * kcols
    vtasks = (32 if esize == 2 else 64) * kcols
    rows = [c // kcols for c in range(kchunks)]
    cols = [c % kcols for c in range(kchunks)]
    assert max(rows) == 63 and max(cols) * 16 + 16 == d * esize
    assert sorted(zip(rows, cols)) == [(i, j) for i in range(64) for j in range(kcols)]
    vrows = [(p // kcols) * (2 if esize == 2 else 1) for p in range(vtasks)]
    assert max(vrows) + (1 if esize == 2 else 0) == 63
    for b in range(tps):
        if P["ndim"] == 2:
            cx, cy = b // nby, b % nby
            cells = [(ux, uy) for ux in range(cx - 1, cx + 2) for uy in range(cy - 1, cy + 2)
                     if 0 <= ux < nbx and 0 <= uy < nby]
            csz = r * r
            nnear = (len(cells) * csz + KT - 1) // KT
            got = []
            for t in range(nnear):
                for row in range(KT):
                    pg = t * KT + row
                    ci = pg // csz
                    if ci >= len(cells):
                        continue
                    p = pg - ci * csz
                    ux, uy = cells[ci]
                    got.append((ux * r + p // r) * side + uy * r + p % r)
            want = sorted((ux * r + a) * side + uy * r + c for ux, uy in cells for a in range(r) for c in range(r))
        else:
            lo = (b - 1) * r if b > 0 else 0
            hi = min((b + 1) * r if causal else (b + 2) * r, n)
            nnear = (hi - lo + KT - 1) // KT
            got = [lo + t * KT + row for t in range(nnear) for row in range(KT) if lo + t * KT + row < hi]
            want = list(range(lo, hi))
        assert all(0 <= x < n for x in got), ("near row outside the slice", b)
        assert sorted(got) == want, ("near tiles do not cover the near field once", b)
        nloads += 2 * nnear
    if P["nslot"]:
        rows = _coarse_rows(P, "2d" if P["ndim"] == 2 else "1d", qt)
        assert ((rows == -1) | ((rows >= 0) & (rows < R))).all()
        nloads += 2 * ((P["nslot"] + KT - 1) // KT) * tps
    return nloads * P["nslice"]


def check_plan(P, grids=(1, 3, 8, 9, 100, 1024, 2048, 4096, 8192)):
    """Every check that applies to the plan's forward pass."""
    geom = "2d" if P["ndim"] == 2 else "1d"
    if small_blocks(P):
        return check_generic_issue(P), None
    loads = check_attend_issue(P, geom, grids=grids)
    if P.get("pair2d"):
        loads = check_pair_issue(P, grids=grids)
    staged = None
    if P["nsets"] > 0 and P["dtype"] == 1 and P["depth"] > 0:
        staged = check_coarsen2d_stream(P) if geom == "2d" else check_coarsen1d_stream(P)
    return loads, staged
