// attend.hip -- fused multilevel FMA attention (Eq. fma1d / Eq. fma2d) on gfx950.
//
// One workgroup owns one query tile: a base block of r queries (1D) or an
// r x r cell (2D), 32 queries per wave.  It walks a list of 64-row key
// tiles: the near-field tiles (blocks b-1 .. b+1 in 1D, the 3x3 cells in 2D,
// their tokens packed 64 to a tile) and then the interaction-list tiles,
// whose rows are gathered coarse keys and values (3 slots per level in 1D,
// 27 in 2D, empty slots masked).  All tiles feed ONE online softmax
// (running max and sum per query), so the score matrix is never stored.
// Blocks smaller than a wave (1D r = 16 or 32, 2D 4 x 4 cells) take one
// wave whose lanes past the block compute on a repeated query and store
// nothing; their near field is not a whole number of tiles, so the rows
// past it are masked like empty coarse slots.
//
// Matrix-core mapping (wave64, MFMA 32x32):
//   S^T = K_tile Q^T   A = 32 keys x 16 d from LDS, B = Q^T held in registers
//   O^T += V^T P^T     A = V^T from a transposed LDS copy, B = P^T taken
//                      straight from the S^T accumulators (no LDS round trip)
// In the S^T accumulator a lane owns one query column (lane & 31) and 16 of
// the 32 key rows, so the row max / row sum of the softmax need one
// cross-lane exchange (lane ^ 32) per tile and the running max, sum and
// rescale factor are per-lane scalars.  The key order inside a 16-key MFMA
// step is permuted identically on the A and B side, which leaves the
// contraction unchanged.
//
// bf16 path: v_mfma_f32_32x32x16_bf16, fp32 accumulation.
// fp32 path: v_mfma_f32_32x32x2_f32, all arithmetic in fp32.
// Tiles are double-staged: the next tile's global loads are in flight while
// the current tile is multiplied out of LDS.
#include "fma_device.hpp"
#include "fma_kernels.hpp"

namespace fma_dev {

namespace {

constexpr int KT = 64;      // keys per tile
constexpr int KPB = 72;     // LDS pitch (bf16) of V^T rows (64 keys + 8)

// LDS pitch of a K (and fp32 V) row of D channels: D + 8 bf16 or D + 4 fp32
// elements (16-byte aligned rows that start on different banks)
template <bool BF16, int D>
constexpr int kRowPitch = BF16 ? D + 8 : D + 4;

template <bool BF16, int D>
struct TileSmem;
template <int D>
struct TileSmem<true, D> {
    __bf16 k[KT * kRowPitch<true, D>];
    __bf16 vt[D * KPB];
    int valid[KT];
};
template <int D>
struct TileSmem<false, D> {
    float k[KT * kRowPitch<false, D>];
    float v[KT * kRowPitch<false, D>];
    int valid[KT];
};

// The coarse-set tables the tile loads index by a computed set, copied to
// LDS once per workgroup (indexing the argument block with a computed index
// makes the compiler copy the whole block to scratch).
struct LvTab {
    int lvl[kMaxSets], M[kMaxSets], My[kMaxSets], off[kMaxSets];
};

// Where the rows of the key tiles of one query tile come from.
struct TileMap {
    int nnear;          // near-field tiles
    long long klo;      // 1D / dense: first near key
    long long khi;      // 1D / dense: one past the last near key
    int ncell;          // 2D: near cells, the in-map 3x3 window row-major:
    int wx0, wy0, wny;  // cell ci is (wx0 + ci / wny, wy0 + ci % wny)
    int csz;            // 2D: tokens per cell (r * r); near row p is token p % csz of cell p / csz
    bool partial;       // the last near tile holds rows past the near field
    int qb, cx, cy;     // query block (1D) / cell (2D)
};

// Element offset of tile row `row` of tile `t`, or -1 for an empty slot.
// *coarse tells whether the offset indexes the coarse arrays.
template <int GEOM, int D>
__device__ inline long long row_source(const AttnArgs &a, const LvTab &lt, const TileMap &m, int slice, int t,
                                       int row, bool *coarse)
{
    if (t < m.nnear) {
        *coarse = false;
        long long tok;
        if constexpr (GEOM == GEOM_2D) {
            const int pg = t * KT + row;   // position in the near cells' tokens, cell after cell
            const int ci = pg / m.csz;
            if (ci >= m.ncell) return -1;
            const int wr = ci / m.wny;
            const int ncx = m.wx0 + wr, ncy = m.wy0 + ci - wr * m.wny;
            const int p = pg - ci * m.csz;
            const int pa = p / a.r, pb = p - pa * a.r;
            tok = (long long)(ncx * a.r + pa) * a.side + (ncy * a.r + pb);
        } else {
            tok = m.klo + (long long)t * KT + row;
            if (tok >= m.khi) return -1;
        }
        return ((long long)slice * a.n + tok) * D;
    }
    *coarse = true;
    // slot = level * slot_group + basis * K + j; slots past the bases of a
    // level (per-level padding) and past the list are empty
    const int kslot = (GEOM == GEOM_2D) ? kSlots2D : kSlots1D;
    const int slot = (t - m.nnear) * KT + row;
    if (slot >= a.nslot) return -1;
    const int lev = slot / a.slot_group, rem = slot - lev * a.slot_group;
    const int b = rem / kslot, j = rem - b * kslot;
    if (b >= a.rank) return -1;
    const int set = lev * a.rank + b;
    int g;
    if constexpr (GEOM == GEOM_2D)
        g = list2d_entry(m.cx, m.cy, lt.lvl[set], j, lt.M[set], lt.My[set]);
    else
        g = list1d_entry(m.qb, lt.lvl[set], j, lt.M[set], a.causal);
    if (g < 0) return -1;
    return ((long long)slice * a.R + lt.off[set] + g) * D;
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Printed per-level normalisation of one 32-key block of coarse scores x
// (log2 units, masked slots -inf): the keys form aligned groups of grp (4, 8,
// 16 or 32) slots, one level each; element i of a lane holds key row
// 8 * (i >> 2) + 4 * hh + (i & 3), so a group is 1 chunk of 4 in-lane (grp 4),
// that chunk in both lanes of the pair lane, lane ^ 32 (8), two chunks (16) or
// all four (32).  Each key's weight becomes lnear * exp2(x - m_g) / l_g, with
// m_g and l_g the group's own maximum and sum; an empty group gives 0.
__device__ inline void level_weights(f32x16 &x, float lnear, int grp)
{
    float cm[4], cl[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) cm[c] = fmaxf(fmaxf(x[4 * c], x[4 * c + 1]), fmaxf(x[4 * c + 2], x[4 * c + 3]));
    if (grp >= 16) {
        cm[0] = cm[1] = fmaxf(cm[0], cm[1]);
        cm[2] = cm[3] = fmaxf(cm[2], cm[3]);
    }
    if (grp >= 32) cm[0] = cm[1] = cm[2] = cm[3] = fmaxf(cm[0], cm[2]);
    if (grp >= 8) {
#pragma unroll
        for (int c = 0; c < 4; ++c) cm[c] = fmaxf(cm[c], __shfl_xor(cm[c], 32));
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        cm[c] = cm[c] > -INFINITY ? cm[c] : 0.0f;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[4 * c + e] = fast_exp2(x[4 * c + e] - cm[c]);
        cl[c] = (x[4 * c] + x[4 * c + 1]) + (x[4 * c + 2] + x[4 * c + 3]);
    }
    if (grp >= 16) {
        cl[0] = cl[1] = cl[0] + cl[1];
        cl[2] = cl[3] = cl[2] + cl[3];
    }
    if (grp >= 32) cl[0] = cl[1] = cl[2] = cl[3] = cl[0] + cl[2];
    if (grp >= 8) {
#pragma unroll
        for (int c = 0; c < 4; ++c) cl[c] += __shfl_xor(cl[c], 32);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const float f = cl[c] > 0.0f ? lnear / cl[c] : 0.0f;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[4 * c + e] *= f;
    }
}

// LIN (FMA-linear, query downsampling): a coarse slot of level l is scored
// with the coarse query of the block's own level-l group (the same for every
// query of the block) instead of the query itself; the slot scores of a
// coarse tile are formed once per workgroup, one slot per thread.
// WIDE: per-level normalisation with levels of several 32-key blocks (2D,
// rank p >= 2), the only plans that need the level accumulators.
template <bool BF16, int NW, int GEOM, bool LIN, int D, bool WIDE>
__global__ __launch_bounds__(64 * NW) void attend_kernel(AttnArgs a)
{
    constexpr int NT = 64 * NW;
    constexpr int ND = D / 32;                    // 32-channel blocks of O (accumulators)
    constexpr int KP = kRowPitch<BF16, D>;        // LDS pitch of K (and fp32 V) rows
    static_assert(D == 32 || D == 64 || D == 128, "head dim");
    __shared__ TileSmem<BF16, D> sm;
    __shared__ LvTab lt;
    __shared__ float lin_q[LIN ? kMaxCoarse * D : 1];          // coarse query of each level
    __shared__ float lin_s[LIN ? KT : 1];                      // raw scores of a coarse tile's slots

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int hh = lane >> 5, l32 = lane & 31;

    // coarse-set tables into LDS (one thread per set; read after the barrier)
    for (int e = tid; e < a.lv.nlev && e < kMaxSets; e += NT) {
        lt.lvl[e] = a.lv.lvl[e];
        lt.M[e] = a.lv.M[e];
        lt.My[e] = a.lv.My[e];
        lt.off[e] = a.lv.off[e];
    }
    __syncthreads();

    // Consecutive workgroup ids go round-robin over the 8 XCDs; remap so
    // that neighbouring query tiles (which share near-field K/V) land on
    // the same XCD and its L2.
    int wg = blockIdx.x;
    const int total = gridDim.x;
    if ((total & 7) == 0) {
        const int per = total >> 3;
        wg = (wg & 7) * per + (wg >> 3);
    }
    const int slice = wg / a.tiles_per_slice;
    const int qt = wg - slice * a.tiles_per_slice;

    TileMap m;
    m.qb = qt;
    m.cx = m.cy = 0;
    m.ncell = 0;
    m.wx0 = m.wy0 = 0;
    m.wny = 1;
    m.csz = 1;
    m.klo = 0;
    m.khi = 0;
    if constexpr (GEOM == GEOM_2D) {
        m.cx = qt / a.nby;
        m.cy = qt - m.cx * a.nby;
        m.csz = a.r * a.r;
        m.wx0 = m.cx > 0 ? m.cx - 1 : 0;
        m.wy0 = m.cy > 0 ? m.cy - 1 : 0;
        const int wx1 = m.cx + 1 < a.nbx ? m.cx + 1 : m.cx, wy1 = m.cy + 1 < a.nby ? m.cy + 1 : m.cy;
        m.wny = wy1 - m.wy0 + 1;
        m.ncell = (wx1 - m.wx0 + 1) * m.wny;
        m.nnear = (m.ncell * m.csz + KT - 1) / KT;
        m.partial = (m.ncell * m.csz) % KT != 0;
    } else if constexpr (GEOM == GEOM_1D) {
        const long long lo = qt > 0 ? (long long)(qt - 1) * a.r : 0;
        long long hi = a.causal ? (long long)(qt + 1) * a.r : (long long)(qt + 2) * a.r;
        if (hi > a.n) hi = a.n;
        m.klo = lo;
        m.khi = hi;
        m.nnear = (int)((hi - lo + KT - 1) / KT);
        m.partial = (hi - lo) % KT != 0;
    } else {
        long long hi = a.causal ? (long long)(qt + 1) * a.qtile : a.n;
        if (hi > a.n) hi = a.n;
        m.khi = hi;
        m.nnear = (int)((hi + KT - 1) / KT);
        m.partial = hi % KT != 0;
    }
    const int ntiles = m.nnear + (GEOM == GEOM_DENSE ? 0 : a.ncoarse_tiles);

    // This lane's query (lanes past a block smaller than the wave repeat one
    // of its queries and store nothing).
    const bool qlive = wave * 32 + l32 < a.qtile;
    const int ql = qlive ? wave * 32 + l32 : l32 % a.qtile;
    long long qtok;
    if constexpr (GEOM == GEOM_2D) {
        const int pa = ql / a.r, pb = ql - pa * a.r;
        qtok = (long long)(m.cx * a.r + pa) * a.side + (m.cy * a.r + pb);
    } else {
        qtok = (long long)qt * a.qtile + ql;
    }
    const long long qrow = ((long long)slice * a.n + qtok) * D;
    // largest query index of this wave (1D / dense), for skipping masked tiles
    const long long wave_qmax = (long long)qt * a.qtile + wave * 32 + 31;

    // Q^T operand, resident for the whole tile loop.
    bf16x8 qb[BF16 ? D / 16 : 1];
    float qf[BF16 ? 1 : D / 2];
    if constexpr (BF16) {
        const __bf16 *qp = static_cast<const __bf16 *>(a.q) + qrow;
#pragma unroll
        for (int c = 0; c < D / 16; ++c) qb[c] = *reinterpret_cast<const bf16x8 *>(qp + 16 * c + 8 * hh);
    } else {
        const float *qp = static_cast<const float *>(a.q) + qrow;
#pragma unroll
        for (int c = 0; c < D / 2; ++c) qf[c] = qp[2 * c + hh];
    }

    // ---------------------------------------------------------------- loads
    // bf16: K = 64 rows x D/8 chunks of 16 B; V = 32 key pairs x D/8 chunks.
    // fp32: K and V = 64 rows x D/4 chunks of 16 B each.
    constexpr int KCOLS = BF16 ? D / 8 : D / 4;    // 16-byte chunks per row
    constexpr int KCHUNKS = KT * KCOLS;
    constexpr int VTASKS = BF16 ? (KT / 2) * KCOLS : KT * KCOLS;
    constexpr int KPER = (KCHUNKS + NT - 1) / NT;
    constexpr int VPER = (VTASKS + NT - 1) / NT;
    uint4 kreg[KPER];
    int kval[KPER];
    uint4 vreg[VPER][BF16 ? 2 : 1];

    const __bf16 *kb16 = nullptr;
    auto fetch = [&](int t) {
#pragma unroll
        for (int i = 0; i < KPER; ++i) {
            const int c = tid + i * NT;
            kreg[i] = make_uint4(0, 0, 0, 0);
            kval[i] = 0;
            if (c < KCHUNKS) {
                const int row = c / KCOLS, col = c - row * KCOLS;
                bool co;
                const long long off = row_source<GEOM, D>(a, lt, m, slice, t, row, &co);
                if (off >= 0) {
                    const char *base = static_cast<const char *>(co ? a.kbar : a.k);
                    kreg[i] = *reinterpret_cast<const uint4 *>(base + (off * (BF16 ? 2 : 4)) + col * 16);
                    kval[i] = 1;
                }
            }
        }
#pragma unroll
        for (int i = 0; i < VPER; ++i) {
            const int p = tid + i * NT;
#pragma unroll
            for (int e = 0; e < (BF16 ? 2 : 1); ++e) vreg[i][e] = make_uint4(0, 0, 0, 0);
            if (p < VTASKS) {
                if constexpr (BF16) {
                    const int kp = p / KCOLS, col = p - kp * KCOLS;
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        bool co;
                        const long long off = row_source<GEOM, D>(a, lt, m, slice, t, 2 * kp + e, &co);
                        if (off >= 0) {
                            const char *base = static_cast<const char *>(co ? a.vbar : a.v);
                            vreg[i][e] = *reinterpret_cast<const uint4 *>(base + off * 2 + col * 16);
                        }
                    }
                } else {
                    const int row = p / KCOLS, col = p - row * KCOLS;
                    bool co;
                    const long long off = row_source<GEOM, D>(a, lt, m, slice, t, row, &co);
                    if (off >= 0) {
                        const char *base = static_cast<const char *>(co ? a.vbar : a.v);
                        vreg[i][0] = *reinterpret_cast<const uint4 *>(base + off * 4 + col * 16);
                    }
                }
            }
        }
    };
    (void)kb16;

    auto stash = [&]() {
#pragma unroll
        for (int i = 0; i < KPER; ++i) {
            const int c = tid + i * NT;
            if (c < KCHUNKS) {
                const int row = c / KCOLS, col = c - row * KCOLS;
                if constexpr (BF16)
                    *reinterpret_cast<uint4 *>(&sm.k[row * KP + col * 8]) = kreg[i];
                else
                    *reinterpret_cast<uint4 *>(&sm.k[row * KP + col * 4]) = kreg[i];
                if (col == 0) sm.valid[row] = kval[i];
            }
        }
#pragma unroll
        for (int i = 0; i < VPER; ++i) {
            const int p = tid + i * NT;
            if (p < VTASKS) {
                if constexpr (BF16) {
                    // transpose a pair of keys x 8 channels into V^T[d][key]
                    const int kp = p / KCOLS, col = p - kp * KCOLS;
                    const uint32_t aw[4] = {vreg[i][0].x, vreg[i][0].y, vreg[i][0].z, vreg[i][0].w};
                    const uint32_t bw[4] = {vreg[i][1].x, vreg[i][1].y, vreg[i][1].z, vreg[i][1].w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t lo = __builtin_amdgcn_perm(bw[e], aw[e], 0x05040100u);
                        const uint32_t hi = __builtin_amdgcn_perm(bw[e], aw[e], 0x07060302u);
                        const int d = col * 8 + 2 * e;
                        *reinterpret_cast<uint32_t *>(&sm.vt[d * KPB + 2 * kp]) = lo;
                        *reinterpret_cast<uint32_t *>(&sm.vt[(d + 1) * KPB + 2 * kp]) = hi;
                    }
                } else {
                    const int row = p / KCOLS, col = p - row * KCOLS;
                    *reinterpret_cast<uint4 *>(&sm.v[row * KP + col * 4]) = vreg[i][0];
                }
            }
        }
    };

    // ------------------------------------------------------------- softmax
    float mrun = -1.0e30f;   // running max (log2 units), finite so that exp2 of differences is safe
    float lrun = 0.f;        // this lane's half of the running sum
    f32x16 o[ND];
#pragma unroll
    for (int db = 0; db < ND; ++db) o[db] = f32x16{0};

    if constexpr (LIN) {
        // coarse query of the block's own group at every level (rank 1: set = level)
        const long long lim = (long long)a.nslice * a.R * D;
        for (int idx = tid; idx < a.lv.nlev * D; idx += NT) {
            const int lev = idx / D, c = idx - (idx / D) * D;
            long long g;
            if constexpr (GEOM == GEOM_2D)
                g = (long long)(m.cx >> lev) * lt.My[lev] + (m.cy >> lev);
            else
                g = m.qb >> lev;
            const long long e = ((long long)slice * a.R + lt.off[lev] + g) * D + c;
            float x = 0.f;
            if (e >= 0 && e < lim) {
                if constexpr (BF16)
                    x = static_cast<float>(static_cast<const __bf16 *>(a.qbar)[e]);
                else
                    x = static_cast<const float *>(a.qbar)[e];
            }
            lin_q[idx] = x;
        }
    }

    // O^T += V^T P^T for 32-key block kb of the staged tile, the weights p
    // in accumulator layout (element i is key row 8 * (i >> 2) + 4 * hh + (i & 3))
    auto pv_block = [&](const f32x16 &p, int kb, f32x16 (&acc)[ND]) {
        if constexpr (BF16) {
            // P^T operand of each 16-key step straight from the accumulators
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                bf16x8 pb;
#pragma unroll
                for (int e = 0; e < 8; ++e) pb[e] = static_cast<__bf16>(p[8 * hf + e]);
                const int base = kb * 32 + 16 * hf + 4 * hh;
#pragma unroll
                for (int db = 0; db < ND; ++db) {
                    const int d = db * 32 + l32;
                    const bf16x4 lo = *reinterpret_cast<const bf16x4 *>(&sm.vt[d * KPB + base]);
                    const bf16x4 hi = *reinterpret_cast<const bf16x4 *>(&sm.vt[d * KPB + base + 8]);
                    const bf16x8 av = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                    acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb, acc[db], 0, 0, 0);
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int kr = kb * 32 + (i >> 2) * 8 + 4 * hh + (i & 3);
#pragma unroll
                for (int db = 0; db < ND; ++db)
                    acc[db] = __builtin_amdgcn_mfma_f32_32x32x2f32(sm.v[kr * KP + db * 32 + l32], p[i], acc[db], 0,
                                                                   0, 0);
            }
        }
    };
    // per-level normalisation with levels wider than a 32-key block (2D rank
    // p >= 2): the open level's own online softmax -- max ml, this lane's
    // half of the sum ll, accumulators ol -- added to O as
    // lnear * O_level / l_level after the level's last block
    f32x16 ol[WIDE ? ND : 1];
#pragma unroll
    for (int db = 0; db < (WIDE ? ND : 1); ++db) ol[db] = f32x16{0};
    float ml = -INFINITY, ll = 0.f;

    fetch(0);
    for (int t = 0; t < ntiles; ++t) {
        __syncthreads();
        stash();
        __syncthreads();
        if (t + 1 < ntiles) fetch(t + 1);

        const bool near_tile = t < m.nnear;
        long long key0 = 0;
        if constexpr (GEOM != GEOM_2D) {
            key0 = m.klo + (long long)t * KT;
            // causal: a near tile wholly after this wave's queries adds nothing
            if (near_tile && a.causal && key0 > wave_qmax) continue;
        }

        f32x16 s[2];
        s[0] = f32x16{0};
        s[1] = f32x16{0};
        if constexpr (BF16) {
#pragma unroll
            for (int c = 0; c < D / 16; ++c) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb) {
                    const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(&sm.k[(kb * 32 + l32) * KP + 16 * c + 8 * hh]);
                    s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[c], s[kb], 0, 0, 0);
                }
            }
        } else {
#pragma unroll
            for (int c = 0; c < D / 2; ++c) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb) {
                    const float ka = sm.k[(kb * 32 + l32) * KP + 2 * c + hh];
                    s[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(ka, qf[c], s[kb], 0, 0, 0);
                }
            }
        }

        if constexpr (LIN) {
            if (!near_tile) {
                // slot scores with the coarse queries, one slot per thread
                constexpr int K = GEOM == GEOM_2D ? kSlots2D : kSlots1D;
                if (tid < KT) {
                    float dot = 0.f;
                    const int slot = (t - m.nnear) * KT + tid;
                    const int set = slot / K;
                    if (sm.valid[tid] && set < a.lv.nlev) {
                        for (int c = 0; c < D; ++c) {
                            if constexpr (BF16)
                                dot += static_cast<float>(sm.k[tid * KP + c]) * lin_q[set * D + c];
                            else
                                dot += sm.k[tid * KP + c] * lin_q[set * D + c];
                        }
                    }
                    lin_s[tid] = dot;
                }
                __syncthreads();
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) s[kb][i] = lin_s[kb * 32 + (i >> 2) * 8 + 4 * hh + (i & 3)];
            }
        }

        // scale, mask, tile max
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int kr = kb * 32 + (i >> 2) * 8 + 4 * hh + (i & 3);
                bool ok;
                if (GEOM != GEOM_2D && near_tile)
                    ok = (!a.causal || (key0 + kr) <= qtok) && (!m.partial || sm.valid[kr] != 0);
                else if (near_tile)
                    ok = !m.partial || sm.valid[kr] != 0;
                else
                    ok = sm.valid[kr] != 0;
                const float x = ok ? s[kb][i] * a.scale_log2 : -INFINITY;
                s[kb][i] = x;
                mx = fmaxf(mx, x);
            }
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        if constexpr (WIDE) {
            if (!near_tile) {
                const float lnear = lrun + __shfl_xor(lrun, 32);
    #pragma unroll
                for (int kb = 0; kb < 2; ++kb) {
                    const int s0 = (t - m.nnear) * KT + kb * 32;   // first slot of the block
                    if (s0 >= a.nslot) break;
                    if (s0 % a.slot_group == 0) {
    #pragma unroll
                        for (int db = 0; db < ND; ++db) ol[db] = f32x16{0};
                        ml = -INFINITY;
                        ll = 0.f;
                    }
                    float bm = -INFINITY;
    #pragma unroll
                    for (int i = 0; i < 16; ++i) bm = fmaxf(bm, s[kb][i]);
                    bm = fmaxf(bm, __shfl_xor(bm, 32));
                    const float mnew = fmaxf(ml, bm);
                    // (a slot is empty for every query alike, so this is uniform;
                    // the ballot keeps the matrix-core step out of a divergent branch)
                    if (__builtin_amdgcn_ballot_w64(mnew > -INFINITY) != 0) {
                        const float mref = mnew > -INFINITY ? mnew : 0.f;
                        const float corr = ml > -INFINITY ? fast_exp2(ml - mref) : 0.f;   // ol, ll are 0 until then
                        ml = mnew;
                        ll *= corr;
    #pragma unroll
                        for (int i = 0; i < 16; ++i) {
    #pragma unroll
                            for (int db = 0; db < ND; ++db) ol[db][i] *= corr;
                            const float p = fast_exp2(s[kb][i] - mref);
                            s[kb][i] = p;
                            ll += p;
                        }
                        pv_block(s[kb], kb, ol);
                    }
                    if ((s0 + 32) % a.slot_group == 0 || s0 + 32 >= a.nslot) {
                        const float lsum = ll + __shfl_xor(ll, 32);
                        const float f = lsum > 0.f ? lnear / lsum : 0.f;
    #pragma unroll
                        for (int i = 0; i < 16; ++i) {
    #pragma unroll
                            for (int db = 0; db < ND; ++db) o[db][i] += f * ol[db][i];
                        }
                    }
                }
                continue;
            }
        }
        if (a.norm_level && !near_tile) {
            // printed per-level normalisation: the near tiles are done, so m
            // and the row sum are the near field's; each level is normalised
            // on its own and weighted by that row sum
            const float lnear = lrun + __shfl_xor(lrun, 32);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) level_weights(s[kb], lnear, a.slot_group);
        } else {
            const float mnew = fmaxf(mrun, mx);
            const float corr = fast_exp2(mrun - mnew);
            mrun = mnew;
            lrun *= corr;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
#pragma unroll
                for (int db = 0; db < ND; ++db) o[db][i] *= corr;
            }
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float p = fast_exp2(s[kb][i] - mnew);
                    s[kb][i] = p;
                    lrun += p;
                }
        }

#pragma unroll
        for (int kb = 0; kb < 2; ++kb) pv_block(s[kb], kb, o);
    }

    // ----------------------------------------------------------- epilogue
    const float ltot = lrun + __shfl_xor(lrun, 32);
    const float inv = 1.0f / ltot;
    if (!qlive) return;
#pragma unroll
    for (int db = 0; db < ND; ++db) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int d = db * 32 + g * 8 + 4 * hh;
            const float x0 = o[db][4 * g] * inv, x1 = o[db][4 * g + 1] * inv;
            const float x2 = o[db][4 * g + 2] * inv, x3 = o[db][4 * g + 3] * inv;
            if constexpr (BF16) {
                uint2 w = make_uint2(pack_bf16x2(x0, x1), pack_bf16x2(x2, x3));
                *reinterpret_cast<uint2 *>(static_cast<__bf16 *>(a.out) + qrow + d) = w;
            } else {
                *reinterpret_cast<float4 *>(static_cast<float *>(a.out) + qrow + d) = make_float4(x0, x1, x2, x3);
            }
        }
    }
}

template <bool BF16, int GEOM, bool LIN, int D, bool WIDE>
hipError_t launch_nw_w(const AttnArgs &a, hipStream_t st)
{
    const unsigned grid = (unsigned)a.tiles_per_slice * (unsigned)a.nslice;
    if (a.qtile <= 0 || a.qtile > 256 || (a.qtile > 32 && a.qtile % 32)) return hipErrorInvalidValue;
    switch ((a.qtile + 31) / 32) {
    case 1: hipLaunchKernelGGL((attend_kernel<BF16, 1, GEOM, LIN, D, WIDE>), dim3(grid), dim3(64), 0, st, a); break;
    case 2: hipLaunchKernelGGL((attend_kernel<BF16, 2, GEOM, LIN, D, WIDE>), dim3(grid), dim3(128), 0, st, a); break;
    case 4: hipLaunchKernelGGL((attend_kernel<BF16, 4, GEOM, LIN, D, WIDE>), dim3(grid), dim3(256), 0, st, a); break;
    case 6: hipLaunchKernelGGL((attend_kernel<BF16, 6, GEOM, LIN, D, WIDE>), dim3(grid), dim3(384), 0, st, a); break;
    case 8: hipLaunchKernelGGL((attend_kernel<BF16, 8, GEOM, LIN, D, WIDE>), dim3(grid), dim3(512), 0, st, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <bool BF16, int GEOM, bool LIN, int D>
hipError_t launch_nw_d(const AttnArgs &a, hipStream_t st)
{
    // levels of several 32-key blocks: 2D per-level plans of rank >= 2
    if constexpr (GEOM == GEOM_2D && !LIN)
        if (a.norm_level && a.slot_group > 32) return launch_nw_w<BF16, GEOM, LIN, D, true>(a, st);
    return launch_nw_w<BF16, GEOM, LIN, D, false>(a, st);
}

template <bool BF16, int GEOM, bool LIN>
hipError_t launch_nw(const AttnArgs &a, hipStream_t st)
{
    switch (a.head_dim) {
    case 32: return launch_nw_d<BF16, GEOM, LIN, 32>(a, st);
    case 64: return launch_nw_d<BF16, GEOM, LIN, 64>(a, st);
    case 128: return launch_nw_d<BF16, GEOM, LIN, 128>(a, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_attend(const AttnArgs &a, bool bf16, int geometry, hipStream_t st)
{
    if (a.nslice == 0 || a.tiles_per_slice == 0) return hipSuccess;
    if (a.qbar) {   // FMA-linear
        if (geometry == GEOM_DENSE) return hipErrorInvalidValue;
        if (bf16) return geometry == GEOM_1D ? launch_nw<true, GEOM_1D, true>(a, st) : launch_nw<true, GEOM_2D, true>(a, st);
        return geometry == GEOM_1D ? launch_nw<false, GEOM_1D, true>(a, st) : launch_nw<false, GEOM_2D, true>(a, st);
    }
    if (bf16) {
        if (geometry == GEOM_1D) return launch_nw<true, GEOM_1D, false>(a, st);
        if (geometry == GEOM_2D) return launch_nw<true, GEOM_2D, false>(a, st);
        return launch_nw<true, GEOM_DENSE, false>(a, st);
    }
    if (geometry == GEOM_1D) return launch_nw<false, GEOM_1D, false>(a, st);
    if (geometry == GEOM_2D) return launch_nw<false, GEOM_2D, false>(a, st);
    return launch_nw<false, GEOM_DENSE, false>(a, st);
}

}  // namespace fma_dev
