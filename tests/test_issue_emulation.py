"""Host-side emulation of the kernels' address arithmetic (tests/issue_emulation.py)
for every shape the GPU tests and the benchmark launch, driven by the
library's own plans (fma_plan_params): the fused attention's tile stream and
the streaming coarsening's rows, weights, staging and outputs stay in bounds
and cover what they must.  Runs on the CPU; nothing touches a device."""
import itertools
import zlib

import numpy as np
import pytest

import fma_inputs
import issue_emulation as emu
import paper_2310_11960_amd as F


def _params(ndim, causal, dt, B, H, size, r, rank=1, per_level=False, linear=False, head_dim=64):
    """size: 1D n; 2D the side of a square map or (rows, columns)."""
    if ndim == 1:
        op = F.FMA(ndim=1, batch=B, heads=H, seq_len=size, block=r, causal=causal, head_dim=head_dim,
                   dtype=fma_inputs.custom("x", 1, causal, dt).torch_dtype, rank=rank,
                   norm=F.FMA_NORM_PER_LEVEL if per_level else F.FMA_NORM_JOINT, linear=linear)
    else:
        rows, cols = size if isinstance(size, tuple) else (size, size)
        op = F.FMA(ndim=2, batch=B, heads=H, seq_len=rows * cols, side=cols, block=r, head_dim=head_dim,
                   dtype=fma_inputs.custom("x", 2, False, dt, side=8, block=8).torch_dtype, rank=rank,
                   norm=F.FMA_NORM_PER_LEVEL if per_level else F.FMA_NORM_JOINT, linear=linear)
    return F.fma_plan_params(op.handle)


def _workload_case(name):
    per_level = name.endswith("_level")
    base, _, p = name.replace("_level", "").partition("_p")
    w = fma_inputs.WORKLOADS[base]
    size = w.side if w.ndim == 2 else w.n
    return (w.ndim, w.causal, w.dtype, w.batch, w.heads, size, w.block, int(p) if p else 1, per_level)


WORKLOAD_NAMES = ["C1", "C2", "C3", "C4", "C5", "C3_p4", "C4_p4", "C5_p4", "C3_level", "C4_level", "C5_level",
                  "C4_p4_level", "C5_p4_level"]

# rectangular 2D maps: (rows, columns) -- wide, tall, ragged on both axes, a
# single row of cells, odd cell columns (no cell pairs), every cell side, rank
# and per-level
RECT_SHAPES = [
    (2, False, "bf16", 1, 2, (32, 64), 8, 1, False), (2, False, "bf16", 1, 2, (128, 32), 8, 1, False),
    (2, False, "f32", 1, 2, (24, 40), 8, 1, False), (2, False, "bf16", 1, 1, (40, 24), 8, 1, False),
    (2, False, "bf16", 1, 2, (64, 128), 16, 1, False), (2, False, "bf16", 1, 2, (16, 64), 4, 1, False),
    (2, False, "bf16", 1, 2, (8, 64), 8, 1, False), (2, False, "bf16", 1, 1, (96, 64), 8, 3, False),
    (2, False, "bf16", 1, 2, (32, 64), 8, 1, True), (2, False, "f32", 1, 1, (48, 16), 4, 1, False),
    (2, False, "bf16", 1, 1, (64, 8), 8, 1, False), (2, False, "bf16", 2, 2, (96, 160), 8, 1, False),
    (2, False, "bf16", 1, 2, (256, 64), 8, 1, False), (2, False, "bf16", 1, 2, (64, 128), 16, 2, False),
    (2, False, "bf16", 1, 1, (8, 96), 8, 1, False), (2, False, "bf16", 1, 2, (16, 128), 4, 1, False),
    (2, False, "f32", 1, 1, (64, 8), 8, 1, False), (2, False, "f32", 1, 1, (16, 40), 4, 1, True),
    (2, False, "bf16", 2, 2, (32, 64), 8, 1, False), (2, False, "bf16", 1, 2, (40, 24), 8, 1, False),
    # 2D per-level at rank p >= 2 (levels of whole 32-slot blocks)
    (2, False, "bf16", 1, 2, 64, 8, 2, True), (2, False, "f32", 1, 1, 40, 8, 3, True),
    (2, False, "bf16", 1, 2, 64, 16, 4, True), (2, False, "bf16", 1, 1, 32, 4, 2, True),
    (2, False, "bf16", 1, 1, 64, 8, 5, True), (2, False, "bf16", 1, 2, 128, 8, 3, True),
    (2, False, "bf16", 1, 2, (32, 64), 8, 2, True), (2, False, "f32", 1, 1, 32, 4, 2, True),
    (2, False, "bf16", 1, 4, 128, 8, 2, True),
]

SHAPES = [
    # ndim, causal, dtype, B, H, n / side, r, rank, per_level -- the GPU tests' shapes
    (1, False, "f32", 1, 2, 1024, 64, 1, False), (1, True, "f32", 1, 2, 1024, 64, 1, False),
    (1, False, "bf16", 2, 2, 4096, 128, 1, False), (1, True, "bf16", 2, 2, 4096, 128, 1, False),
    (1, False, "bf16", 1, 3, 64 * 23, 64, 1, False), (1, True, "bf16", 1, 3, 64 * 21, 64, 1, False),
    (1, True, "f32", 1, 1, 128 * 11, 128, 1, False), (1, False, "bf16", 1, 2, 192 * 10, 192, 1, False),
    (1, True, "bf16", 1, 2, 256 * 8, 256, 1, False), (1, False, "bf16", 1, 2, 64, 64, 1, False),
    (1, True, "f32", 1, 2, 128, 64, 1, False), (2, False, "bf16", 2, 2, 64, 8, 1, False),
    (2, False, "f32", 1, 2, 32, 8, 1, False), (2, False, "bf16", 1, 2, 64, 16, 1, False),
    (2, False, "bf16", 1, 2, 40, 8, 1, False), (2, False, "f32", 1, 1, 80, 16, 1, False),
    (2, False, "bf16", 1, 1, 8, 8, 1, False), (1, False, "bf16", 1, 2, 2048, 64, 4, False),
    (1, True, "bf16", 1, 2, 16384, 128, 4, False), (1, True, "f32", 1, 2, 1024, 64, 3, False),
    (1, False, "f32", 1, 1, 64 * 23, 64, 5, False), (1, True, "bf16", 1, 2, 64 * 21, 64, 2, False),
    (1, False, "bf16", 1, 1, 65536, 128, 8, False), (2, False, "bf16", 1, 2, 64, 8, 4, False),
    (2, False, "bf16", 1, 1, 128, 8, 5, False), (2, False, "f32", 1, 1, 40, 8, 5, False),
    (2, False, "bf16", 1, 1, 64, 16, 3, False), (1, False, "f32", 1, 2, 1024, 64, 1, True),
    (1, True, "bf16", 2, 2, 4096, 128, 1, True), (1, True, "bf16", 1, 3, 64 * 21, 64, 1, True),
    (1, False, "f32", 1, 1, 128 * 11, 128, 1, True), (1, False, "bf16", 1, 2, 2048, 64, 2, True),
    (1, True, "f32", 1, 2, 1024, 64, 3, True), (1, True, "bf16", 1, 2, 16384, 128, 4, True),
    (1, False, "bf16", 1, 1, 2048, 64, 10, True), (1, False, "bf16", 1, 2, 256 * 8, 256, 1, True),
    (2, False, "bf16", 2, 2, 64, 8, 1, True), (2, False, "f32", 1, 1, 40, 8, 1, True),
    (2, False, "bf16", 1, 2, 64, 16, 1, True),
    # coarsening cases
    (1, False, "bf16", 2, 3, 64 * 23, 64, 1, False), (2, False, "bf16", 1, 2, 128, 8, 1, False),
    (2, False, "f32", 1, 2, 88, 8, 1, False), (2, False, "bf16", 1, 1, 256, 8, 1, False),
    (1, True, "bf16", 4, 8, 4096, 64, 4, False), (1, False, "f32", 1, 2, 64 * 23, 64, 3, False),
    (1, False, "bf16", 1, 2, 128 * 37, 128, 5, False), (2, False, "bf16", 1, 2, 128, 8, 4, False),
    (2, False, "f32", 1, 1, 88, 8, 5, False), (1, False, "bf16", 1, 2, 16384, 128, 4, False),
    (2, False, "bf16", 1, 2, 128, 8, 5, False), (2, False, "bf16", 1, 2, 128, 16, 2, False),
    (2, False, "bf16", 2, 2, 32, 8, 1, False),
    # peaked structure cases
    (1, True, "bf16", 1, 4, 64 * 45, 64, 1, False), (1, False, "bf16", 1, 4, 256 * 16, 256, 1, False),
    (1, True, "bf16", 1, 2, 192 * 12, 192, 1, False), (1, False, "bf16", 1, 4, 16384, 128, 4, False),
    (1, True, "bf16", 1, 4, 8192, 64, 4, False), (1, True, "bf16", 1, 4, 8192, 128, 1, True),
    (2, False, "bf16", 1, 4, 128, 16, 1, False), (2, False, "bf16", 1, 4, 8 * 13, 8, 1, False),
    (2, False, "bf16", 1, 4, 128, 8, 1, True),
    # backward and no-alloc shapes (their forward and coarsening)
    (1, False, "bf16", 2, 2, 1024, 64, 1, False), (1, True, "bf16", 1, 2, 2048, 128, 1, False),
    (1, False, "bf16", 1, 1, 64 * 11, 64, 1, False), (1, True, "bf16", 1, 1, 1536, 192, 2, False),
    (2, False, "bf16", 1, 1, 40, 8, 2, False), (1, False, "bf16", 2, 4, 8192, 128, 1, False),
    # rank and size extremes: 64 coarse sets in 1D, 16 in 2D, a long sequence
    (1, False, "bf16", 1, 1, 4096, 64, 10, False), (1, True, "bf16", 2, 2, 1 << 20, 128, 4, False),
    (2, False, "bf16", 1, 1, 256, 8, 3, False),
    # blocks smaller than a wave (the register-staged kernel)
    (1, False, "bf16", 1, 2, 1024, 16, 1, False), (1, True, "bf16", 1, 2, 16 * 37, 16, 1, False),
    (1, False, "f32", 1, 2, 32 * 23, 32, 2, False), (1, True, "f32", 1, 1, 1024, 32, 1, True),
    (2, False, "bf16", 1, 2, 64, 4, 1, False), (2, False, "f32", 1, 1, 44, 4, 1, True),
    (2, False, "bf16", 1, 1, 32, 4, 3, False), (1, False, "bf16", 2, 2, 16 * 37, 16, 1, False),
    (1, False, "bf16", 2, 2, 4096, 16, 1, False), (1, False, "f32", 1, 2, 32 * 45, 32, 3, False),
    (2, False, "bf16", 1, 2, 128, 4, 1, False), (2, False, "f32", 1, 2, 44, 4, 1, False),
    (2, False, "bf16", 1, 1, 64, 4, 4, False), (1, True, "bf16", 1, 4, 16 * 45, 16, 1, False),
    (1, False, "bf16", 1, 2, 4096, 32, 2, False), (2, False, "bf16", 1, 4, 44, 4, 1, False),
    (1, True, "bf16", 1, 3, 16 * 37, 16, 1, False), (1, False, "bf16", 1, 2, 16, 16, 1, False),
    (2, False, "bf16", 1, 1, 4, 4, 1, False), (1, True, "bf16", 1, 2, 4096, 32, 2, False),
    # rectangular maps (rows, columns)
] + RECT_SHAPES


def _ids(c):
    size = "%dx%d" % c[5] if isinstance(c[5], tuple) else str(c[5])
    return "%dd_%s_%s_B%dH%d_%s_r%d_p%d%s" % (c[0], "causal" if c[1] else "bidi", c[2], c[3], c[4], size, c[6],
                                            c[7], "_level" if c[8] else "")


@pytest.mark.parametrize("name", WORKLOAD_NAMES)
def test_workload_addresses(name):
    c = _workload_case(name)
    P = _params(*c)
    loads, staged = emu.check_plan(P)
    assert loads > 0


@pytest.mark.parametrize("case", SHAPES, ids=[_ids(c) for c in SHAPES])
def test_shape_addresses(case):
    P = _params(*case)
    emu.check_plan(P, grids=(1, 5, 8, 1024))


# head dims 32 and 128 (the GPU tests' shapes): the register-staged kernel
HEADDIM_SHAPES = [
    (1, False, "bf16", 2, 2, 1024, 64, 1, False, 32), (1, True, "bf16", 1, 2, 4096, 128, 1, False, 128),
    (1, False, "f32", 1, 2, 1024, 64, 1, False, 128), (1, True, "f32", 1, 2, 16 * 37, 16, 1, False, 32),
    (1, False, "bf16", 1, 3, 64 * 23, 64, 1, False, 128), (1, True, "bf16", 1, 1, 256 * 8, 256, 1, False, 128),
    (1, False, "bf16", 1, 2, 32 * 45, 32, 3, False, 32), (1, False, "bf16", 1, 2, 4096, 64, 4, False, 128),
    (1, True, "bf16", 1, 2, 2048, 64, 2, True, 32), (2, False, "bf16", 1, 2, 64, 8, 1, False, 128),
    (2, False, "bf16", 1, 2, 32, 4, 1, False, 32), (2, False, "f32", 1, 1, 44, 4, 1, False, 128),
    (2, False, "bf16", 1, 2, 64, 16, 1, False, 128), (2, False, "bf16", 1, 2, 64, 8, 2, True, 128),
    (2, False, "f32", 1, 2, (24, 40), 8, 1, False, 32), (2, False, "bf16", 1, 2, (32, 64), 8, 2, False, 128),
    (1, False, "f32", 1, 2, 2048, 128, 1, False, 32),
]


@pytest.mark.parametrize("case", HEADDIM_SHAPES, ids=[_ids(c[:9]) + "_d%d" % c[9] for c in HEADDIM_SHAPES])
def test_head_dim_addresses(case):
    P = _params(*case[:9], head_dim=case[9])
    assert P["head_dim"] == case[9] and emu.small_blocks(P) and not P["pair2d"] and P["depth"] == 0
    emu.check_plan(P, grids=(1, 5, 8, 1024))


@pytest.mark.parametrize("name", ["C4", "C5"])
def test_linear_plan_addresses(name):
    w = fma_inputs.WORKLOADS[name]
    P = _params(w.ndim, False, w.dtype, w.batch, w.heads, w.side if w.ndim == 2 else w.n, w.block, linear=True)
    emu.check_plan(P, grids=(1, 1024))


@pytest.mark.parametrize("n,causal", [(1024, False), (4096, True), (65536, False)])
def test_dense_reference_addresses(n, causal):
    P = _params(1, causal, "bf16", 1, 2, n, 64)
    emu.check_attend_issue(P, "1d", dense=True, grids=(1, 8, 1024))


@pytest.mark.parametrize("Mx,My", [(1, 1), (2, 3), (5, 7), (8, 8), (9, 4), (3, 12)])
def test_list2d_inverse(Mx, My):
    """The backward reduction finds the list entry naming a coarse square in
    closed form; it agrees with list2d_entry for every group and square."""
    for lvl in (1, 2, 3):
        span = 1 << (lvl - 1)
        for qx in range(Mx):
            for qy in range(My):
                named = {}
                for j in range(27):
                    gi = int(emu.list2d_entry(np.array(qx * span), np.array(qy * span), lvl, j, Mx, My))
                    if gi >= 0:
                        named[gi] = j
                for u in range(Mx):
                    for v in range(My):
                        assert emu.list2d_slot_of(qx, qy, u, v) == named.get(u * My + v, -1), (qx, qy, u, v)


def test_closed_form_lists_match_the_oracle():
    """The emulator's list arithmetic is the kernel's closed form: it equals
    the oracle's set-builder lists (so the coarse rows checked above are the
    right ones, not only in bounds)."""
    import numpy as np

    import oracle
    for n, r, causal in ((1024, 64, False), (64 * 23, 64, True), (4096, 128, True)):
        ref, _, _ = oracle.lists_1d(n, r, kcap=3)
        nb = n // r
        L = oracle.num_levels(nb)
        b = np.arange(nb)
        for l in range(1, L):
            M = -(-n // (r << (l - 1)))
            got = np.stack([emu.list1d_entry(b, l, j, M, causal) for j in range(3)], 1)
            for bb in range(nb):
                want = [g for g in ref[bb, l - 1] if g >= 0]
                if causal:
                    s = r << (l - 1)
                    want = [g for g in want if min((g + 1) * s, n) - 1 <= bb * r]
                assert sorted(g for g in got[bb] if g >= 0) == want
    for Hm, W, r in ((64, 64, 8), (40, 40, 8), (64, 64, 16), (24, 72, 8), (96, 32, 8), (8, 64, 8), (48, 16, 4)):
        ref = oracle.lists_2d(W, r, kcap=27, H=Hm)
        nbx, nby = Hm // r, W // r
        L = oracle.num_levels(max(nbx, nby))
        cells = np.arange(nbx * nby)
        for l in range(1, L):
            M, My = -(-Hm // (r << (l - 1))), -(-W // (r << (l - 1)))
            got = np.stack([emu.list2d_entry(cells // nby, cells % nby, l, j, M, My) for j in range(27)], 1)
            for c in cells:
                assert sorted(g for g in got[c] if g >= 0) == [g for g in ref[c, l - 1] if g >= 0]


def test_emulator_catches_planted_plan_mistakes():
    """Mistakes planted in a copy of a real plan (never in a kernel) are
    caught: coarse rows past the slice, a list slot of a set that does not
    exist, a coarsening unit that is not a multiple of the narrowest group, a
    ring that does not fit its LDS, a near field that is not whole tiles."""
    import copy

    base = _params(1, False, "bf16", 2, 2, 65536, 128)
    planted = []
    p = copy.deepcopy(base)
    p["R"] -= 1                                  # one coarse row short
    planted.append(("R", p))
    p = copy.deepcopy(base)
    p["nslot"] += 3                              # slots of a ninth set
    planted.append(("nslot", p))
    p = copy.deepcopy(base)
    p["chunk"] = 192                             # unit not r * 2^k
    p["nchunk"] = -(-p["n"] // 192)
    planted.append(("chunk", p))
    p = copy.deepcopy(base)
    p["wave_lds"] -= 64                          # ring + staging does not fit
    planted.append(("wave_lds", p))
    p = copy.deepcopy(base)
    p["npartial"] -= 1                           # partial rows of one set too few
    planted.append(("npartial", p))
    p = copy.deepcopy(base)
    p["sets"][3]["off"] = p["R"] - 2             # a set's rows run past the slice
    planted.append(("set off", p))
    p = copy.deepcopy(base)
    p["block"], p["qtile"] = 96, 96              # near field of 1.5 tiles
    p["tiles_per_slice"] = p["n"] // 96
    planted.append(("block", p))
    q2 = _params(2, False, "bf16", 1, 1, 128, 8)
    p = copy.deepcopy(q2)
    p["sets"][2]["M"] += 1                       # a square past the map
    planted.append(("2d M", p))
    q3 = _params(2, False, "bf16", 1, 1, (32, 128), 8)
    p = copy.deepcopy(q3)
    p["sets"][2]["My"] += 1                      # a column of squares past the map
    planted.append(("2d My", p))
    p = copy.deepcopy(q3)
    p["nby"], p["nbx"] = p["nbx"], p["nby"]      # cells counted along the wrong axis
    planted.append(("2d axes", p))
    for what, P in planted:
        with pytest.raises(AssertionError):
            emu.check_plan(P, grids=(8,))
        # the unplanted plans pass
    emu.check_plan(base, grids=(8,))
    emu.check_plan(q2, grids=(8,))
    emu.check_plan(q3, grids=(8,))
