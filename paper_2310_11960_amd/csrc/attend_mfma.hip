// attend_mfma.hip -- fused multilevel FMA attention for bf16 on gfx950
// (Eq. fma1d / Eq. fma2d under one softmax per query).
//
// One workgroup owns one query tile: a base block of r queries (1D) or an
// r x r cell (2D), 32 queries per wave.  It walks a list of 64-key tiles:
// first the near field (blocks b-1 .. b+1 in 1D, the 3x3 cells in 2D), then
// the interaction-list tiles whose rows are coarse keys/values gathered from
// the per-level arrays (3 slots per level in 1D, 27 in 2D, empty slots
// masked).  All tiles feed one online softmax, so scores never leave
// registers.
//
// Data movement.  K and V tiles go from HBM/L2 straight into LDS with
// 16-byte direct-to-LDS loads (no VGPR staging), double-buffered: the next
// tile is in flight while the current one is multiplied, one barrier per
// tile.  Rows are 128 bytes (64 bf16 channels) and the eight 16-byte chunks
// of each row are XOR-swizzled so that both read patterns below are free of
// bank conflicts:
//   K: chunk c of row r sits at chunk position c ^ ((r & 7) ^ ((r >> 3) & 1))
//   V: chunk c of row r sits at chunk position c ^ (2 * (r & 3))
//
// Matrix cores (wave64, v_mfma_f32_32x32x16_bf16, fp32 accumulation):
//   S^T = K Q^T    A = 32 keys x 16 channels (ds_read_b128 of K rows),
//                  B = Q^T, resident in registers for the whole loop
//   O^T += V^T P^T A = V^T read with the transposing LDS load
//                  ds_read_b64_tr_b16 from the row-major V tile,
//                  B = P^T taken from the S^T accumulators as they are.
// In the S^T accumulator a lane owns one query (lane & 31) and 16 of the 32
// keys of a block, so the softmax reductions are in-lane plus one exchange
// with lane ^ 32 (v_permlane32_swap).  The key order inside each 16-key PV
// step is permuted identically on the A and B sides.
//
// Softmax.  Scores are scaled inside the exponent: p = exp2(s * c - m) with
// c = tau * log2(e).  The running maximum m is only raised when a tile's
// maximum exceeds it by more than 8 (in log2 units), so p <= 2^8 and the
// accumulators are rescaled rarely; the result is the same softmax, since
// numerator and denominator share the reference m.
//
// Printed per-level normalisation (norm_level).  The near tiles come first,
// so when the coarse tiles start the near field's m and row sum l are final.
// Each level's slots then form one aligned group of 4, 8, 16 or 32 keys of a
// 32-key block; a coarse key j of level g gets the weight
// l * exp2(s_j - m_g) / l_g (m_g, l_g: the group's own maximum and sum), so
// that the final O / l adds each level's own softmax average to the near
// field's.
#include "fma_device.hpp"
#include "fma_kernels.hpp"

namespace fma_dev {

namespace {

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void gbl_void;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

#ifndef FMA_NS_WIDE
#define FMA_NS_WIDE 3     // LDS stages for workgroups of four or more waves
#endif
#ifndef FMA_NS_NARROW
#define FMA_NS_NARROW 2   // LDS stages for two-wave workgroups
#endif
constexpr int KT = 64;             // keys per tile
constexpr int ROWB = 128;          // bytes of one bf16 row (64 channels)
constexpr int TILEB = KT * ROWB;   // one K or V tile, 8 KB
constexpr int MAX_CTILES = 7;      // coarse tiles: ceil(27 * 16 / 64)
constexpr int MAX_SLOTS = MAX_CTILES * KT;
static_assert(MAX_SLOTS == kMaxSlotTable, "slot table size");

template <int NS, int SLOTS>
struct Smem {
    unsigned char k[NS][TILEB];
    unsigned char v[NS][TILEB];
    int crow[2][SLOTS];                // coarse slot -> coarse row (-1: empty), two blocks
    unsigned long long cmask[NS];      // slot validity bits of the coarse tile in each stage
    int lv_m[kMaxSets];                // groups of each coarse set's level (2D: rows of squares)
    int lv_my[kMaxSets];               // 2D: columns of squares of each set's level
    int lv_off[kMaxSets];              // first coarse row of each set
    int lv_lvl[kMaxSets];              // level of each set
};

// 16-byte direct-to-LDS load: lane L's 16 bytes from gptr land at LDS byte
// lds_base + 16 * L.  Issued as inline assembly so that the compiler does not
// treat later LDS reads of the other buffer as waiting on it; the loop
// waits for its own loads explicitly (vmcnt) before the tile barrier.
__device__ inline void dma16(const void *gptr, uint32_t lds_base)
{
    asm volatile("global_load_lds_dwordx4 %0, off" : : "v"(gptr), "{m0}"(lds_base) : "memory");
}

// Same with a scalar base and a 32-bit lane offset (no immediate offset: on
// these loads it would move the LDS destination as well).
__device__ inline void dma16_sv(uint32_t voff, const void *sbase, uint32_t lds_base)
{
    // the base is the same in every lane: make that visible to the compiler
    // (readfirstlane returns a signed int: widen each half as unsigned)
    const uint64_t b = reinterpret_cast<uint64_t>(sbase);
    const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32)));
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b)));
    const uint64_t u = (static_cast<uint64_t>(hi) << 32) | lo;
    asm volatile("global_load_lds_dwordx4 %0, %1" : : "v"(voff), "s"(reinterpret_cast<const void *>(u)),
                 "{m0}"(lds_base) : "memory");
}

// Wait until at most N of this wave's vector-memory operations are in
// flight (loads complete in issue order), leaving LDS and export counters.
template <int N>
__device__ inline void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ inline uint32_t lds_addr(const void *p)
{
    return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_void *)p));
}

__device__ inline int swz_k(int row) { return (row & 7) ^ ((row >> 3) & 1); }
__device__ inline int swz_v(int row) { return 2 * (row & 3); }

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// max of x over this lane and lane ^ 32
__device__ inline float max_pair(float x)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ inline float sum_pair(float x)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ inline uint32_t pack_bf16(float lo, float hi)
{
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 p = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
    return __builtin_bit_cast(uint32_t, p);
}

enum TileMask { MASK_NONE = 0, MASK_CAUSAL = 1, MASK_SLOTS = 2 };

// Scores of one 32-key block for the wave's 32 queries (lane & 31), in
// log2 units relative to the reference maximum m:
//   S'^T = K (c Q)^T + C,  C = -m in every element,
// so p = exp2(S') needs no per-score arithmetic besides the exponential.
// The four K fragments are read from LDS together, so that the MFMA chain
// waits on LDS once rather than before every step.
__device__ __attribute__((always_inline)) inline f32x16 block_scores(const unsigned char *kt, const int (&koff)[4],
                                                                     const bf16x8 (&qb)[4], const f32x16 &cneg)
{
    f32x16 sc = cneg;
    bf16x8 ka[4];
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) ka[c4] = *reinterpret_cast<const bf16x8 *>(kt + koff[c4]);
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[c4], qb[c4], sc, 0, 0, 0);
    return sc;
}

// Softmax and P V of one block whose scores sc come from block_scores.
//   MASK_CAUSAL: block row kr is visible iff kr <= lim (lim already holds
//                the query position minus the row offset of this lane);
//   MASK_SLOTS : block row kr is visible iff bit 8 * (i >> 2) + (i & 3) of
//                the lane's slot mask word is set (coarse tiles).
// `first` marks the wave's first block, which sets m to that block's maximum.
// FIRST (a fully visible first block, the first near tile) does that without
// the general rescale: m, O and l start from this block alone, the PV MFMAs
// of its first half take zero C operands and no accumulator is zeroed first.
template <int MASK, bool FIRST = false>
__device__ __attribute__((always_inline)) inline void block_softmax_pv(
    f32x16 sc, const unsigned char *vt, const int (&voff)[2], int lim, uint32_t mword, bool first, f32x16 &o0,
    f32x16 &o1, f32x16 &cneg, float &m, float &l)
{
    if constexpr (MASK == MASK_CAUSAL) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
            if ((i >> 2) * 8 + (i & 3) > lim) sc[i] = -INFINITY;
    } else if constexpr (MASK == MASK_SLOTS) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
            if (!((mword >> ((i >> 2) * 8 + (i & 3))) & 1u)) sc[i] = -INFINITY;
    }

    // The reference maximum m only has to keep the weights 2^(s - m) finite:
    // fp32 and bf16 share the exponent range, so scores may exceed m by a lot
    // before anything overflows, and O / l does not depend on m.  m is set
    // from the wave's first block; after that a block takes no maximum: each
    // half-block's weights are checked, and only when they sum past 2^64 in
    // some lane (a score above m + 60) is m raised to the maximum of the
    // scores not yet consumed, O and l rescaled and the half redone (rare).
    // Each query decides for itself -- other lanes shift by 0 and scale by
    // exp2(0) = 1 exactly -- so a row never depends on the other rows of the
    // wave.  (`first` is the same in every lane of the wave.)
    // in-lane maximum of elements lo .. 15, then with lane ^ 32
    auto tail_max = [&](int lo) {
        float t[5];
#pragma unroll
        for (int j = 0; j < 5; ++j)
            t[j] = fmaxf(fmaxf(3 * j >= lo ? sc[3 * j] : -INFINITY, 3 * j + 1 >= lo ? sc[3 * j + 1] : -INFINITY),
                         3 * j + 2 >= lo ? sc[3 * j + 2] : -INFINITY);
        return max_pair(fmaxf(fmaxf(fmaxf(t[0], t[1]), t[2]), fmaxf(fmaxf(t[3], t[4]), sc[15])));
    };
    if constexpr (FIRST) {
        // the wave's first block, every key visible: m starts at its maximum
        // and O, l start from this block alone (zero C operands below)
        const float mx = tail_max(0);
        m = mx;
        l = 0.0f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            cneg[i] = -mx;
            sc[i] -= mx;
        }
    } else if (first) {
        // a first block that may be partly masked: m from its visible maximum
        // (none visible: m stays); O and l are still 0
        float step = tail_max(0);
        if (!(step > -INFINITY)) step = 0.0f;
        m += step;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            cneg[i] -= step;
            sc[i] -= step;
        }
    }

    // P^T operand straight from the accumulator, row sum of the bf16 weights
    // (v_dot2 with (1, 1)), O^T += V^T P^T
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
        uint32_t w[4];
        float lh = 0.0f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            w[e] = pack_bf16(fast_exp2(sc[8 * hf + 2 * e]), fast_exp2(sc[8 * hf + 2 * e + 1]));
            lh = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, lh, false);
        }
        if constexpr (!FIRST) {
            if (__builtin_expect(__builtin_amdgcn_ballot_w64(lh > 0x1p64f) != 0, 0)) {
                const float mx = tail_max(8 * hf);
                const float step = mx > 0.0f ? mx : 0.0f;
                const float corr = fast_exp2(-step);
                m += step;
                l *= corr;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    cneg[i] -= step;
                    sc[i] -= step;
                    o0[i] *= corr;
                    o1[i] *= corr;
                }
                lh = 0.0f;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    w[e] = pack_bf16(fast_exp2(sc[8 * hf + 2 * e]), fast_exp2(sc[8 * hf + 2 * e + 1]));
                    lh = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, lh, false);
                }
            }
        }
        l += lh;
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 pw = {w[0], w[1], w[2], w[3]};
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
        const int kbase = hf * 16 * ROWB;
#pragma unroll
        for (int db = 0; db < 2; ++db) {
            const s16x4 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(vt + kbase + voff[db]));
            const s16x4 r2 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(vt + kbase + 8 * ROWB + voff[db]));
            typedef short s16x8 __attribute__((ext_vector_type(8)));
            const s16x8 av = {r1[0], r1[1], r1[2], r1[3], r2[0], r2[1], r2[2], r2[3]};
            const bf16x8 va = __builtin_bit_cast(bf16x8, av);
            const f32x16 zc = {0};
            if (db == 0)
                o0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, FIRST && hf == 0 ? zc : o0, 0, 0, 0);
            else
                o1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, FIRST && hf == 0 ? zc : o1, 0, 0, 0);
        }
    }
}

// One block on its own (masked and coarse tiles): scores, softmax, P V.
template <int MASK>
__device__ __attribute__((always_inline)) inline void attend_block(
    const unsigned char *kt, const unsigned char *vt, const int (&koff)[4], const int (&voff)[2],
    const bf16x8 (&qb)[4], int lim, uint32_t mword, bool first, f32x16 &o0, f32x16 &o1, f32x16 &cneg,
    float &m, float &l)
{
    block_softmax_pv<MASK>(block_scores(kt, koff, qb, cneg), vt, voff, lim, mword, first, o0, o1, cneg, m, l);
}

// One coarse block under the printed per-level normalisation: the block's
// keys form aligned groups of grp (4, 8, 16 or 32) slots, one level each.  In
// the S^T accumulator element i of a lane holds key row
// 8 * (i >> 2) + 4 * hh + (i & 3), so a group of 4 is one in-lane chunk of
// 4 elements, a group of 8 is that chunk in both lanes of the pair (lane and
// lane ^ 32), 16 two chunks and 32 all of them.  Each key gets
// lnear * exp2(s - m_g) / l_g; an empty group (every slot masked) gives 0.
// m and the row sum stay the near field's.
__device__ __attribute__((always_inline)) inline void block_levels_pv(
    f32x16 sc, const unsigned char *vt, const int (&voff)[2], uint32_t mword, float lnear, int grp, f32x16 &o0,
    f32x16 &o1)
{
#pragma unroll
    for (int i = 0; i < 16; ++i)
        if (!((mword >> ((i >> 2) * 8 + (i & 3))) & 1u)) sc[i] = -INFINITY;
    float cm[4], cl[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) cm[c] = fmaxf(fmaxf(sc[4 * c], sc[4 * c + 1]), fmaxf(sc[4 * c + 2], sc[4 * c + 3]));
    if (grp >= 16) {
        cm[0] = cm[1] = fmaxf(cm[0], cm[1]);
        cm[2] = cm[3] = fmaxf(cm[2], cm[3]);
    }
    if (grp >= 32) cm[0] = cm[1] = cm[2] = cm[3] = fmaxf(cm[0], cm[2]);
    if (grp >= 8) {
#pragma unroll
        for (int c = 0; c < 4; ++c) cm[c] = max_pair(cm[c]);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        cm[c] = cm[c] > -INFINITY ? cm[c] : 0.0f;   // empty group: every exp2 below is 0
#pragma unroll
        for (int e = 0; e < 4; ++e) sc[4 * c + e] = fast_exp2(sc[4 * c + e] - cm[c]);
        cl[c] = (sc[4 * c] + sc[4 * c + 1]) + (sc[4 * c + 2] + sc[4 * c + 3]);
    }
    if (grp >= 16) {
        cl[0] = cl[1] = cl[0] + cl[1];
        cl[2] = cl[3] = cl[2] + cl[3];
    }
    if (grp >= 32) cl[0] = cl[1] = cl[2] = cl[3] = cl[0] + cl[2];
    if (grp >= 8) {
#pragma unroll
        for (int c = 0; c < 4; ++c) cl[c] = sum_pair(cl[c]);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const float f = cl[c] > 0.0f ? lnear / cl[c] : 0.0f;
#pragma unroll
        for (int e = 0; e < 4; ++e) sc[4 * c + e] *= f;
    }
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = pack_bf16(sc[8 * hf + 2 * e], sc[8 * hf + 2 * e + 1]);
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 pw = {w[0], w[1], w[2], w[3]};
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
        const int kbase = hf * 16 * ROWB;
#pragma unroll
        for (int db = 0; db < 2; ++db) {
            const s16x4 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(vt + kbase + voff[db]));
            const s16x4 r2 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(vt + kbase + 8 * ROWB + voff[db]));
            typedef short s16x8 __attribute__((ext_vector_type(8)));
            const s16x8 av = {r1[0], r1[1], r1[2], r1[3], r2[0], r2[1], r2[2], r2[3]};
            const bf16x8 va = __builtin_bit_cast(bf16x8, av);
            if (db == 0)
                o0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o0, 0, 0, 0);
            else
                o1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o1, 0, 0, 0);
        }
    }
}

// Scalars of the problem the kernel needs, copied out of the argument block.
struct Geo {
    long long n;     // tokens per slice
    int r, side, nbx, nby, qtile, tps, causal;   // nbx, nby: 2D cells along x (rows) and y (columns)
    int nq;          // Q tiles per query block (128 queries each)
    int nctile;      // coarse tiles per query block
    int tpc, lg_r;   // 2D: tiles per cell, log2(r)
};

// One query block: r queries (1D), an r x r cell (2D), two horizontally
// adjacent cells (2D pairs) or qtile queries (dense), and the tiles it
// walks: nq Q tiles, nnear near tiles, nctile coarse tiles (2D pairs: nctile
// for each cell).
struct QBlock {
    int slice, qt, nnear, ntile;
    long long klo;               // 1D / dense: first near key
    int cx, cy, dx0, dy0, ncy;   // 2D: cell and its in-map 3x3 neighbourhood
                                 // 2D pairs: left cell (cx, cy); dx0 as 2D; dy0 = 1 if
                                 // column cy - 1 exists; ncy = columns of the pair's window
};

template <int GEOM>
constexpr bool kIs2D = GEOM == GEOM_2D || GEOM == GEOM_2DP;

template <int GEOM>
__device__ __attribute__((always_inline)) inline QBlock make_qblock(int id, const Geo &g)
{
    QBlock b;
    b.slice = id / g.tps;
    b.qt = id - b.slice * g.tps;
    b.klo = 0;
    b.cx = b.cy = b.dx0 = b.dy0 = 0;
    b.ncy = 1;
    if constexpr (GEOM == GEOM_2DP) {
        // the pair's near window: rows cx-1 .. cx+1, columns cy-1 .. cy+2 in
        // the map, walked column by column: the two shared columns (cy,
        // cy+1), then cy-1 (left cell only), then cy+2 (right cell only)
        const int half = g.nby >> 1;
        b.cx = b.qt / half;
        b.cy = 2 * (b.qt - b.cx * half);
        b.dx0 = b.cx > 0 ? -1 : 0;
        const int dx1 = b.cx + 1 < g.nbx ? 1 : 0;
        b.dy0 = b.cy > 0 ? 1 : 0;
        b.ncy = 2 + b.dy0 + (b.cy + 2 < g.nby ? 1 : 0);
        b.nnear = (dx1 - b.dx0 + 1) * b.ncy * g.tpc;
    } else if constexpr (GEOM == GEOM_2D) {
        b.cx = b.qt / g.nby;
        b.cy = b.qt - b.cx * g.nby;
        b.dx0 = b.cx > 0 ? -1 : 0;
        const int dx1 = b.cx + 1 < g.nbx ? 1 : 0;
        b.dy0 = b.cy > 0 ? -1 : 0;
        const int dy1 = b.cy + 1 < g.nby ? 1 : 0;
        b.ncy = dy1 - b.dy0 + 1;
        b.nnear = (dx1 - b.dx0 + 1) * b.ncy * g.tpc;
    } else if constexpr (GEOM == GEOM_1D) {
        b.klo = b.qt > 0 ? (long long)(b.qt - 1) * g.r : 0;
        long long hi = g.causal ? (long long)(b.qt + 1) * g.r : (long long)(b.qt + 2) * g.r;
        if (hi > g.n) hi = g.n;
        b.nnear = (int)((hi - b.klo) / KT);
    } else {
        long long hi = g.causal ? (long long)(b.qt + 1) * g.qtile : g.n;
        if (hi > g.n) hi = g.n;
        b.nnear = (int)((hi + KT - 1) / KT);
    }
    b.ntile = g.nq + b.nnear + (GEOM == GEOM_2DP ? 2 : 1) * g.nctile;
    return b;
}

// 2D pairs: the near cell of tile-walk cell index ci (column-major over the
// pair's window, columns in the order of make_qblock) and the wave groups
// that use it: bit 0 the left cell's waves (columns cy-1 .. cy+1), bit 1 the
// right cell's (columns cy .. cy+2).
__device__ __attribute__((always_inline)) inline int pair_near_cell(const QBlock &b, int ci, int &ux, int &uy)
{
    const int ncx = b.nnear / b.ncy;   // rows of the window (tiles per cell is 1 for pairs)
    const int cs = ci / ncx, row = ci - cs * ncx;
    ux = b.cx + b.dx0 + row;
    uy = cs < 2 ? b.cy + cs : (cs == 2 && b.dy0) ? b.cy - 1 : b.cy + 2;
    return (uy <= b.cy + 1 ? 1 : 0) | (uy >= b.cy ? 2 : 0);
}

// Token of row p (0 .. qtile-1) of a query block, or of row p of a 2D cell
// (2D pairs: rows 0 .. r*r-1 the left cell, then the right cell).
template <int GEOM>
__device__ __attribute__((always_inline)) inline long long block_token(const QBlock &b, const Geo &g, int p)
{
    if constexpr (GEOM == GEOM_2DP) {
        const int c = p >> (2 * g.lg_r), q = p & ((1 << (2 * g.lg_r)) - 1);
        return (long long)(b.cx * g.r + (q >> g.lg_r)) * g.side + (b.cy + c) * g.r + (q & (g.r - 1));
    } else if constexpr (GEOM == GEOM_2D)
        return (long long)(b.cx * g.r + (p >> g.lg_r)) * g.side + b.cy * g.r + (p & (g.r - 1));
    else
        return (long long)b.qt * g.qtile + p;
}

// Register budget: 1D workgroups of four or more waves are built for four
// waves per SIMD (128 registers) with two LDS stages (36 KB, four workgroups
// per CU), which measured faster than three waves with three stages; 2D and
// dense ones of four or more waves for three (168); two-wave workgroups for
// two (256), which their LDS stages hold to two per SIMD anyway.
#ifndef FMA_WAVES_1D
#define FMA_WAVES_1D 4    // waves per SIMD the 1D kernels of four or more waves are built for
#endif
#ifndef FMA_NS_1D
#define FMA_NS_1D 2       // LDS stages of those 1D kernels
#endif
// (2D pairs under the per-level normalisation keep the levels' own
// accumulators as well: three waves per SIMD, whose register budget holds
// them without spilling)
template <int NW, int GEOM, bool PL = false>
constexpr int kWavesPerEU = NW >= 4 ? (GEOM == GEOM_1D ? FMA_WAVES_1D : GEOM == GEOM_2DP ? (PL ? 3 : 4) : 3) : 2;

// LIN (FMA-linear): every query of a block scores its far field with the
// same coarse queries (its block's own group at each level), so the far
// field of the whole block reduces to one weighted sum: with the slot scores
// s (log2 units), M = max s, Z = sum 2^(s - M) and U = sum 2^(s - M) v_bar.
// The coarse tiles leave the tile stream; lin_far_kernel forms (M, Z, U) of
// every block beforehand and every query folds them into its own (m, l, O)
// before the output.
template <int NW, int GEOM, bool PL, bool LIN>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(kWavesPerEU<NW, GEOM, PL>, kWavesPerEU<NW, GEOM, PL>)))
void attend_mfma_kernel(AttnArgs a)
{
    constexpr int NT = 64 * NW;
    // LDS stages: three (two tiles in flight) when four or more waves share
    // them, two for two-wave workgroups, whose LDS per wave is double.
    constexpr int NS = NW >= 4 ? (GEOM == GEOM_1D ? FMA_NS_1D : GEOM == GEOM_2DP ? 2 : FMA_NS_WIDE) : FMA_NS_NARROW;
    static_assert(GEOM != GEOM_2DP || (NW == 4 && !LIN), "2D pairs: four waves, not FMA-linear");
    constexpr int NLD = 16 / NW;   // fewest of a tile's 16 loads any wave issues
    constexpr int K = kIs2D<GEOM> ? kSlots2D : kSlots1D;
    // slot table: both cells' tables side by side in the paired kernel
    constexpr int SLOTS = GEOM == GEOM_2DP ? kMaxPairSlotTable : MAX_SLOTS;
    __shared__ Smem<NS, SLOTS> sm;
    __shared__ float lin_u[LIN ? kHeadDim + 2 : 1];   // FMA-linear: the block's M, Z, U

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int hh = lane >> 5, l32 = lane & 31;

    Geo g;
    g.n = a.n;
    g.r = a.r;
    g.side = a.side;
    g.nbx = a.nbx;
    g.nby = a.nby;
    g.qtile = GEOM == GEOM_2DP ? 2 * a.qtile : a.qtile;
    g.tps = GEOM == GEOM_2DP ? a.tiles_per_slice / 2 : a.tiles_per_slice;
    g.causal = a.causal;
    g.nq = (NW + 3) / 4;
    g.nctile = LIN ? 0 : (a.nslot + KT - 1) / KT;
    g.tpc = kIs2D<GEOM> ? (a.r * a.r) / KT : 1;
    g.lg_r = 31 - __builtin_clz(a.r);
    const int nslot = a.nslot;

    // ------------------------------------------------ this workgroup's query blocks
    // Workgroups are handed out round-robin over the 8 XCDs.  Each XCD owns
    // one contiguous range of query blocks, which its workgroups walk with a
    // common stride, so the blocks in flight on an XCD are neighbours that
    // read the same near-field K/V from its L2.
    const int total = g.tps * a.nslice;
    const int G = gridDim.x;
    const int nx = G < 8 ? G : 8;
    const int xg = blockIdx.x % nx, jg = blockIdx.x / nx;
    const int gx = (G - 1 - xg) / nx + 1;
    const int blk_end = (int)((long long)total * (xg + 1) / nx);
    const int blk_first = (int)((long long)total * xg / nx) + jg;

    // ------------------------------------------------ per-lane LDS offsets
    // direct loads: lane writes chunk position (lane & 7) of tile row 8i + (lane >> 3)
    const int lrow = lane >> 3;
    const int ldk0 = lrow * ROWB + 16 * ((lane & 7) ^ lrow);            // i even
    const int ldk1 = lrow * ROWB + 16 * ((lane & 7) ^ lrow ^ 1);        // i odd
    const int ldv = lrow * ROWB + 16 * ((lane & 7) ^ (2 * (lrow & 3)));
    // K (and Q) operand reads: row l32 of a 32-row block, logical chunk 2*c4 + hh
    int koff[4];
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) koff[c4] = l32 * ROWB + 16 * ((2 * c4 + hh) ^ swz_k(l32));
    // V^T operand reads (transposing load): see the header comment
    int voff[2];
    {
        const int gq = lane >> 4, s4 = lane & 15, j = s4 >> 2, q = s4 & 3;
        const int row = 4 * (gq >> 1) + j;
#pragma unroll
        for (int db = 0; db < 2; ++db) {
            const int chunk = 4 * db + 2 * (gq & 1) + (q >> 1);
            voff[db] = row * ROWB + 16 * (chunk ^ swz_v(row)) + 8 * (q & 1);
        }
    }

    // coarse slot tables of two consecutive blocks (padding slots stay
    // empty) and the level tables
    for (int t = tid; t < 2 * SLOTS; t += NT) sm.crow[t / SLOTS][t % SLOTS] = -1;
    // one thread per coarse set (indexed loads from the argument block)
    if (tid < a.lv.nlev) {
        sm.lv_m[tid] = a.lv.M[tid];
        sm.lv_my[tid] = a.lv.My[tid];
        sm.lv_off[tid] = a.lv.off[tid];
        sm.lv_lvl[tid] = a.lv.lvl[tid];
    }
    const char *const qg0 = static_cast<const char *>(a.q);
    const char *const kg0 = static_cast<const char *>(a.k);
    const char *const vg0 = static_cast<const char *>(a.v);
    const char *const kbar0 = static_cast<const char *>(a.kbar);
    const char *const vbar0 = static_cast<const char *>(a.vbar);
    const long long Rrows = a.R;
    __syncthreads();

    // ------------------------------------------------ tile issue (direct to LDS)
    // A tile is 16 loads of 8 rows x 128 bytes: loads 0..7 fill the K half of
    // the stage, 8..15 the V half; wave w issues loads w, w + NW, ...  Q
    // tiles carry 128 query rows (64 per half, K swizzle in both).
    QBlock ib = make_qblock<GEOM>(blk_first, g);
    int iblk = blk_first, ilt = 0, ipar = 0;
    bool ivalid = blk_first < blk_end;
    int issued = 0;

    // Slot e of a block's interaction-list table: entry j of basis b of level
    // lev (slot = lev * G + b * K + j).  Joint normalisation: G = K * p, so
    // the set (level, basis) is simply e / K.  Per-level normalisation pads a
    // level's slots to G; the slots past its p bases stay empty.  GI_ =
    // group (or square) index or -1, OFF_ = first coarse row of the set.
    const int sgrp = a.slot_group, rank = a.rank;
#define FMA_SLOT_ENTRY(B_, E_, GI_, OFF_)                                                                        \
    do {                                                                                                         \
        int set_, j_;                                                                                            \
        bool used_ = true;                                                                                       \
        if constexpr (PL) {                                                                                      \
            const int lev_ = (E_) / sgrp, rem_ = (E_) - lev_ * sgrp;                                             \
            const int b_ = rem_ / K;                                                                             \
            j_ = rem_ - b_ * K;                                                                                  \
            set_ = lev_ * rank + b_;                                                                             \
            used_ = b_ < rank;                                                                                   \
        } else {                                                                                                 \
            set_ = (E_) / K;                                                                                     \
            j_ = (E_) - set_ * K;                                                                                \
        }                                                                                                        \
        (GI_) = -1;                                                                                              \
        (OFF_) = 0;                                                                                              \
        if (used_) {                                                                                             \
            const int M_ = sm.lv_m[set_], lvl_ = sm.lv_lvl[set_];                                                \
            (OFF_) = sm.lv_off[set_];                                                                            \
            if constexpr (kIs2D<GEOM>)                                                                           \
                (GI_) = list2d_entry((B_).cx, (B_).cy, lvl_, j_, M_, sm.lv_my[set_]);                            \
            else                                                                                                 \
                (GI_) = list1d_entry((B_).qt, lvl_, j_, M_, g.causal);                                           \
        }                                                                                                        \
    } while (0)

    // 1D: entering a block builds its interaction-list table, every slot at
    // once by wave 0 (the coarse tile that reads it is issued at least one
    // tile barrier later; the two parities keep the table of the block being
    // issued apart from the next one's).
#define FMA_BUILD_LISTS(B_, PAR_)                                                                                \
    do {                                                                                                         \
        if (wave == 0) {                                                                                         \
            for (int e = lane; e < nslot; e += 64) {                                                             \
                int gi, off;                                                                                     \
                FMA_SLOT_ENTRY(B_, e, gi, off);                                                                  \
                sm.crow[PAR_][e] = gi >= 0 ? off + gi : -1;                                                      \
            }                                                                                                    \
        }                                                                                                        \
    } while (0)
    if constexpr (GEOM == GEOM_1D)
        if (ivalid && g.nctile > 0) FMA_BUILD_LISTS(ib, 0);

    // Issue the next tile into stage ST_: 16 loads of 8 rows x 128 bytes,
    // loads 0..7 fill the K half of the stage, 8..15 the V half; wave w
    // issues loads w, w + NW, ...  1D: every load takes a scalar base (the
    // first of its 8 rows) and the lane's 32-bit offset inside those rows.
    // 2D and dense keep per-lane 64-bit addresses and build the list table
    // as a block's first tile is issued (FMA_ISSUE_VGPR).
#define FMA_ISSUE_SCALAR(ST_)                                                                                      \
    do {                                                                                                         \
        const int st_ = (ST_);                                                                                   \
        const uint32_t kdst = __builtin_amdgcn_readfirstlane(lds_addr(sm.k[st_]));                               \
        const uint32_t vdst = __builtin_amdgcn_readfirstlane(lds_addr(sm.v[st_]));                               \
        if (ilt < g.nq) {                                                                                        \
            /* Q tile: 128 query rows (rows past the block repeat harmlessly) */                                 \
            const char *qg = qg0 + (long long)ib.slice * g.n * ROWB;                                             \
            _Pragma("unroll") for (int jj = 0; jj < (16 + NW - 1) / NW; ++jj) {                                  \
                const int j = wave + NW * jj;                                                                    \
                if (j < 16) {                                                                                    \
                    const int i = j & 7, half = j >> 3;                                                          \
                    int p0 = ilt * 128 + half * 64 + 8 * i;                                                      \
                    if (p0 >= g.qtile) p0 -= g.qtile * (p0 / g.qtile);                                           \
                    const long long tok = block_token<GEOM>(ib, g, p0);                                          \
                    dma16_sv((i & 1) ? ldk1 : ldk0, qg + tok * ROWB, (half ? vdst : kdst) + i * 1024);           \
                }                                                                                                \
            }                                                                                                    \
        } else if (ilt < g.nq + ib.nnear) {                                                                      \
            const int t = ilt - g.nq;                                                                            \
            const char *kg = kg0 + (long long)ib.slice * g.n * ROWB;                                             \
            const char *vg = vg0 + (long long)ib.slice * g.n * ROWB;                                             \
            long long tok0 = 0;                                                                                  \
            int ux = 0, uy = 0, sub = 0;                                                                         \
            if constexpr (GEOM == GEOM_2D) {                                                                     \
                const int ci = t / g.tpc;                                                                        \
                sub = t - ci * g.tpc;                                                                            \
                ux = ib.cx + ib.dx0 + ci / ib.ncy;                                                               \
                uy = ib.cy + ib.dy0 + ci % ib.ncy;                                                               \
            } else {                                                                                             \
                tok0 = ib.klo + (long long)t * KT;                                                               \
            }                                                                                                    \
            _Pragma("unroll") for (int jj = 0; jj < (16 + NW - 1) / NW; ++jj) {                                  \
                const int j = wave + NW * jj;                                                                    \
                if (j < 16) {                                                                                    \
                    const int i = j & 7;                                                                         \
                    const bool isv = j >= 8;                                                                     \
                    long long tok;                                                                               \
                    if constexpr (GEOM == GEOM_2D) {                                                             \
                        const int p0 = sub * KT + 8 * i;                                                         \
                        tok = (long long)(ux * g.r + (p0 >> g.lg_r)) * g.side + uy * g.r + (p0 & (g.r - 1));     \
                    } else {                                                                                     \
                        tok = tok0 + 8 * i;                                                                      \
                    }                                                                                            \
                    dma16_sv(isv ? ldv : ((i & 1) ? ldk1 : ldk0), (isv ? vg : kg) + tok * ROWB,                  \
                             (isv ? vdst : kdst) + i * 1024);                                                    \
                }                                                                                                \
            }                                                                                                    \
        } else {                                                                                                 \
            /* coarse tile: gathered rows; empty slots read coarse row 0 (finite, */                             \
            /* weighted by p = 0) and clear their bit in the stage's slot mask */                                \
            const int ct = ilt - g.nq - ib.nnear;                                                                \
            const char *kb_ = kbar0 + (long long)ib.slice * Rrows * ROWB;                                        \
            const char *vb_ = vbar0 + (long long)ib.slice * Rrows * ROWB;                                        \
            _Pragma("unroll") for (int jj = 0; jj < (16 + NW - 1) / NW; ++jj) {                                  \
                const int j = wave + NW * jj;                                                                    \
                if (j < 16) {                                                                                    \
                    const int i = j & 7;                                                                         \
                    const bool isv = j >= 8;                                                                     \
                    int row = sm.crow[ipar][ct * KT + 8 * i + lrow];                                             \
                    if (!isv) {                                                                                  \
                        const unsigned long long bal = __builtin_amdgcn_ballot_w64(row >= 0);                    \
                        if (lane == 0) {                                                                         \
                            uint32_t byte = 0;                                                                   \
                            _Pragma("unroll") for (int rr = 0; rr < 8; ++rr)                                     \
                                byte |= (uint32_t)((bal >> (8 * rr)) & 1ull) << rr;                              \
                            reinterpret_cast<unsigned char *>(&sm.cmask[st_])[i] = (unsigned char)byte;          \
                        }                                                                                        \
                    }                                                                                            \
                    row = row < 0 ? 0 : row;                                                                     \
                    const uint32_t off_ = (uint32_t)row * ROWB + (isv ? ldv : ((i & 1) ? ldk1 : ldk0)) - lrow * ROWB; \
                    dma16_sv(off_, isv ? vb_ : kb_, (isv ? vdst : kdst) + i * 1024);                             \
                }                                                                                                \
            }                                                                                                    \
        }                                                                                                        \
        ++issued;                                                                                                \
        if (++ilt == ib.ntile) {                                                                                 \
            ilt = 0;                                                                                             \
            ipar ^= 1;                                                                                           \
            iblk += gx;                                                                                          \
            ivalid = iblk < blk_end;                                                                             \
            if (ivalid) {                                                                                        \
                ib = make_qblock<GEOM>(iblk, g);                                                                 \
                if (g.nctile > 0) FMA_BUILD_LISTS(ib, ipar);                                                     \
            }                                                                                                    \
        }                                                                                                        \
    } while (0)

#define FMA_ISSUE_VGPR(ST_)                                                                                     \
    do {                                                                                                        \
        const int st = (ST_);                                                                                   \
        const char *kg = kg0 + (long long)ib.slice * g.n * ROWB;                                                \
        const char *vg = vg0 + (long long)ib.slice * g.n * ROWB;                                                \
        if (ilt == 0 && g.nctile > 0) {                                                                         \
/* entering a block: build its interaction-list table (2D pairs: the left */                                    \
/* cell's at slot 0, the right cell's at slot nctile * KT) */                                                   \
            constexpr int NC_ = GEOM == GEOM_2DP ? 2 : 1;                                                       \
            for (int e = tid; e < NC_ * nslot; e += NT) {                                                       \
                const int c_ = e >= nslot ? 1 : 0, el_ = e - c_ * nslot;                                        \
                QBlock cb_ = ib;                                                                                \
                cb_.cy += c_;                                                                                   \
                int gi, off;                                                                                    \
                FMA_SLOT_ENTRY(cb_, el_, gi, off);                                                              \
                sm.crow[ipar][c_ * g.nctile * KT + el_] = gi >= 0 ? off + gi : -1;                              \
            }                                                                                                   \
        }                                                                                                       \
        if (ilt < g.nq) {                                                                                       \
            const char *qg = qg0 + (long long)ib.slice * g.n * ROWB;                                            \
            for (int j = wave; j < 16; j += NW) {                                                               \
                const int i = j & 7, half = j >> 3;                                                             \
                int p0 = ilt * 128 + half * 64 + 8 * i;                                                         \
                if (p0 >= g.qtile) p0 -= g.qtile * (p0 / g.qtile); /* rows past the block: harmless repeats */  \
                const long long tok = block_token<GEOM>(ib, g, p0);                                             \
                const char *src = qg + tok * ROWB + ((i & 1) ? ldk1 : ldk0);                                    \
                unsigned char *dst = (half ? sm.v[st] : sm.k[st]) + i * 1024;                                   \
                dma16(src, __builtin_amdgcn_readfirstlane(lds_addr(dst)));                                      \
            }                                                                                                   \
        } else if (ilt < g.nq + ib.nnear) {                                                                     \
            const int t = ilt - g.nq;                                                                           \
            long long tok0 = 0;                                                                                 \
            int ux = 0, uy = 0, sub = 0;                                                                        \
            if constexpr (GEOM == GEOM_2DP) {                                                                   \
                pair_near_cell(ib, t, ux, uy); /* one tile per 8 x 8 cell */                                    \
            } else if constexpr (GEOM == GEOM_2D) {                                                             \
                const int ci = t / g.tpc;                                                                       \
                sub = t - ci * g.tpc;                                                                           \
                ux = ib.cx + ib.dx0 + ci / ib.ncy;                                                              \
                uy = ib.cy + ib.dy0 + ci % ib.ncy;                                                              \
            } else {                                                                                            \
                tok0 = ib.klo + (long long)t * KT;                                                              \
            }                                                                                                   \
            for (int j = wave; j < 16; j += NW) {                                                               \
                const int i = j & 7;                                                                            \
                const bool isv = j >= 8;                                                                        \
                long long tok;                                                                                  \
                if constexpr (kIs2D<GEOM>) {                                                                    \
                    const int p0 = sub * KT + 8 * i;                                                            \
                    tok = (long long)(ux * g.r + (p0 >> g.lg_r)) * g.side + uy * g.r + (p0 & (g.r - 1));        \
                } else {                                                                                        \
                    tok = tok0 + 8 * i;                                                                         \
                }                                                                                               \
                const char *src = (isv ? vg : kg) + tok * ROWB + (isv ? ldv : ((i & 1) ? ldk1 : ldk0));         \
                unsigned char *dst = (isv ? sm.v[st] : sm.k[st]) + i * 1024;                                    \
                dma16(src, __builtin_amdgcn_readfirstlane(lds_addr(dst)));                                      \
            }                                                                                                   \
        } else {                                                                                                \
/* coarse tile: gathered rows; empty slots read coarse row 0 (finite, */                                        \
/* weighted by p = 0) and clear their bit in the stage's slot mask */                                           \
            const int ct = ilt - g.nq - ib.nnear;                                                               \
            const char *kb_ = kbar0 + (long long)ib.slice * Rrows * ROWB;                                       \
            const char *vb_ = vbar0 + (long long)ib.slice * Rrows * ROWB;                                       \
            for (int j = wave; j < 16; j += NW) {                                                               \
                const int i = j & 7;                                                                            \
                const bool isv = j >= 8;                                                                        \
                int row = sm.crow[ipar][ct * KT + 8 * i + lrow];                                                \
                if (!isv) {                                                                                     \
                    const unsigned long long bal = __builtin_amdgcn_ballot_w64(row >= 0);                       \
                    if (lane == 0) {                                                                            \
                        uint32_t byte = 0;                                                                      \
_Pragma("unroll")                                                                                               \
                        for (int rr = 0; rr < 8; ++rr) byte |= (uint32_t)((bal >> (8 * rr)) & 1ull) << rr;      \
                        reinterpret_cast<unsigned char *>(&sm.cmask[st])[i] = (unsigned char)byte;              \
                    }                                                                                           \
                }                                                                                               \
                row = row < 0 ? 0 : row;                                                                        \
                const char *src = (isv ? vb_ : kb_) + (long long)row * ROWB +                                   \
                                  (isv ? ldv : ((i & 1) ? ldk1 : ldk0)) - lrow * ROWB;                          \
                unsigned char *dst = (isv ? sm.v[st] : sm.k[st]) + i * 1024;                                    \
                dma16(src, __builtin_amdgcn_readfirstlane(lds_addr(dst)));                                      \
            }                                                                                                   \
        }                                                                                                       \
        ++issued;                                                                                               \
        if (++ilt == ib.ntile) {                                                                                \
            ilt = 0;                                                                                            \
            ipar ^= 1;                                                                                          \
            iblk += gx;                                                                                         \
            ivalid = iblk < blk_end;                                                                            \
            if (ivalid) ib = make_qblock<GEOM>(iblk, g);                                                        \
        }                                                                                                       \
    } while (0)

#define FMA_ISSUE_NEXT(ST_)                                                                                      \
    do {                                                                                                         \
        if constexpr (GEOM == GEOM_1D)                                                                           \
            FMA_ISSUE_SCALAR(ST_);                                                                               \
        else                                                                                                     \
            FMA_ISSUE_VGPR(ST_);                                                                                 \
    } while (0)

    // ------------------------------------------------ compute
    // The compute side walks each query block as straight loops -- Q tiles,
    // fully visible near tiles, causal diagonal tiles, coarse tiles -- so that
    // the accumulators O^T, -m and the row sum live in one set of registers
    // throughout (no data-dependent joins except the rare rescale).
    float mrun = 0.f;        // reference maximum (log2 units), set by a block's first scores
    float lrun = 0.f;        // this lane's part of the row sum
    f32x16 o0 = {0}, o1 = {0}, cneg = {0};
    bf16x8 qb[4];
    const float cs = a.scale_log2;
    __bf16 *const outp = static_cast<__bf16 *>(a.out);
    constexpr int BLK = 32 * ROWB;   // bytes of one 32-key block

#pragma unroll
    for (int t0 = 0; t0 < NS - 1; ++t0)
        if (ivalid) FMA_ISSUE_NEXT(t0);

    bool stored = false;   // the previous tile ended a block (8 output stores per wave in flight)
    int step = 0, cst = 0;
    const unsigned char *kt = sm.k[0];
    const unsigned char *vt = sm.v[0];

    // Next compute tile: this wave's loads of it have landed when at most the
    // operations issued after them are outstanding (the loads of the tiles
    // issued later and, after a block ends, its output stores); the barrier
    // makes every wave's loads visible and frees the stage the issue below
    // overwrites.
#define FMA_NEXT_TILE()                                                                                         \
    do {                                                                                                        \
        const int ahead = issued - step - 1 < NS - 2 ? issued - step - 1 : NS - 2;                              \
        if (ahead >= 2)                                                                                         \
            stored ? wait_vmcnt<2 * NLD + 8>() : wait_vmcnt<2 * NLD>();                                         \
        else if (ahead == 1)                                                                                    \
            stored ? wait_vmcnt<NLD + 8>() : wait_vmcnt<NLD>();                                                 \
        else                                                                                                    \
            wait_vmcnt<0>();                                                                                    \
        stored = false;                                                                                         \
        __syncthreads();                                                                                        \
        if (ivalid) FMA_ISSUE_NEXT((step + NS - 1) % NS);                                                       \
        cst = step % NS;                                                                                        \
        kt = sm.k[cst];                                                                                         \
        vt = sm.v[cst];                                                                                         \
        ++step;                                                                                                 \
    } while (0)

    for (int cblk = blk_first; cblk < blk_end; cblk += gx) {
        const QBlock cb = make_qblock<GEOM>(cblk, g);

        // FMA-linear: the block's far field (M, Z, U), formed by lin_far_kernel
        if constexpr (LIN) {
            __syncthreads();   // every wave is done with the previous block's values
            if (tid < kHeadDim + 2) {
                const long long fi = (long long)cblk * (kHeadDim + 2) + tid;
                lin_u[tid] = fi < a.lin_far_elems ? a.lin_far[fi] : 0.f;
            }
            __syncthreads();
        }

        // Q tiles: the waves whose 32 queries a tile holds take their Q^T
        // operand, scaled by tau * log2(e) so that scores come out in log2 units
        for (int qt = 0; qt < g.nq; ++qt) {
            FMA_NEXT_TILE();
            if (wave / 4 == qt) {
                const unsigned char *qt_ = ((wave & 3) >> 1 ? vt : kt) + (wave & 1) * 32 * ROWB;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                    u32x4 w = *reinterpret_cast<const u32x4 *>(qt_ + koff[c]);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        w[e] = pack_bf16(__uint_as_float(w[e] << 16) * cs, __uint_as_float(w[e] & 0xffff0000u) * cs);
                    qb[c] = __builtin_bit_cast(bf16x8, w);
                }
            }
        }
        bool first = true;   // the wave's first block of scores sets m

        // near tiles every query of the block sees in full; the first one
        // starts m, O and l from its own scores (no zeroed accumulators)
        const long long qstart = (long long)cb.qt * g.qtile;   // 1D / dense: first query of the block
        int nfull = cb.nnear;
        if constexpr (!kIs2D<GEOM>)
            if (g.causal) nfull = (int)((qstart - cb.klo) / KT);
        int t = 0;
        if (nfull > 0) {
            FMA_NEXT_TILE();
            const f32x16 zc = {0};
            block_softmax_pv<MASK_NONE, true>(block_scores(kt, koff, qb, zc), vt, voff, 0, 0u, true, o0, o1, cneg,
                                              mrun, lrun);
            attend_block<MASK_NONE>(kt + BLK, vt + BLK, koff, voff, qb, 0, 0u, false, o0, o1, cneg, mrun, lrun);
            first = false;
            t = 1;
        } else {
            mrun = 0.f;
            lrun = 0.f;
            o0 = f32x16{0};
            o1 = f32x16{0};
            cneg = f32x16{0};
        }
        for (; t < nfull; ++t) {
            FMA_NEXT_TILE();
            if constexpr (GEOM == GEOM_2DP) {
                // 2D pairs: the cells of the left column belong to the left
                // cell's waves only, those of the right column to the right
                // cell's (tile 0 is shared)
                int ux_, uy_;
                if (!((pair_near_cell(cb, t, ux_, uy_) >> (wave >> 1)) & 1)) continue;
            }
            attend_block<MASK_NONE>(kt, vt, koff, voff, qb, 0, 0u, first, o0, o1, cneg, mrun, lrun);
            attend_block<MASK_NONE>(kt + BLK, vt + BLK, koff, voff, qb, 0, 0u, false, o0, o1, cneg, mrun, lrun);
            first = false;
        }
        // causal: tiles overlapping the block's own queries; a wave takes the
        // 32-key blocks that start at or before its first query (the one that
        // starts there is its diagonal block, masked to keys <= query)
        const long long wave_q0 = qstart + wave * 32;
        for (int t = nfull; t < cb.nnear; ++t) {
            FMA_NEXT_TILE();
            const long long dq = wave_q0 - (cb.klo + (long long)t * KT);   // a multiple of 32
            const int nsb = dq < 0 ? 0 : (dq >= 32 ? 2 : 1);
            const int lim = (int)dq + l32 - 4 * hh;
#pragma unroll 1
            for (int sb = 0; sb < nsb; ++sb) {
                attend_block<MASK_CAUSAL>(kt + sb * BLK, vt + sb * BLK, koff, voff, qb, lim - 32 * sb, 0u, first,
                                          o0, o1, cneg, mrun, lrun);
                first = false;
            }
        }
        // coarse tiles: gathered interaction-list rows, empty slots masked
        if constexpr (PL) {
            const float lnear = sum_pair(lrun);   // the near field's row sum, final here
            if (kIs2D<GEOM> && sgrp > 32) {
                // 2D rank p >= 2: a level's 27p slots fill sgrp / 32 whole
                // blocks, so each level runs an online softmax of its own
                // (max ml, this lane's half of the sum ll, accumulators
                // ol0/ol1) over its blocks and adds lnear * O_level / l_level
                // to O when its last block is done.  A level's first block
                // with a visible slot sets ml (`first`), so a level whose
                // first blocks are empty still starts from its own maximum.
                f32x16 ol0 = {0}, ol1 = {0}, cl = {0};
                float ml = 0.f, ll = 0.f;
                bool lseen = false;
                // (2D pairs: the left cell's coarse tiles, then the right
                // cell's, each taken by its own waves)
                for (int ct = 0; ct < (GEOM == GEOM_2DP ? 2 : 1) * g.nctile; ++ct) {
                    FMA_NEXT_TILE();
                    int ctl = ct;
                    if constexpr (GEOM == GEOM_2DP) {
                        const int c_ = ct >= g.nctile ? 1 : 0;
                        if (c_ != (wave >> 1)) continue;
                        ctl = ct - c_ * g.nctile;
                    }
                    const unsigned long long mt = sm.cmask[cst];
                    const unsigned long long mlane = mt >> (4 * hh);
                    const int nsb = nslot - ctl * KT > 32 ? 2 : 1;
#pragma unroll 1
                    for (int sb = 0; sb < nsb; ++sb) {
                        const int s0 = ctl * KT + sb * 32;
                        if (s0 % sgrp == 0) {
                            ol0 = f32x16{0};
                            ol1 = f32x16{0};
                            cl = f32x16{0};
                            ml = 0.f;
                            ll = 0.f;
                            lseen = false;
                        }
                        const bool any = ((mt >> (32 * sb)) & 0xffffffffull) != 0;
                        attend_block<MASK_SLOTS>(kt + sb * BLK, vt + sb * BLK, koff, voff, qb, 0,
                                                 (uint32_t)(mlane >> (32 * sb)), !lseen, ol0, ol1, cl, ml, ll);
                        lseen = lseen || any;
                        if ((s0 + 32) % sgrp == 0 || s0 + 32 >= nslot) {
                            const float lsum = sum_pair(ll);
                            const float f = lsum > 0.f ? lnear / lsum : 0.f;
#pragma unroll
                            for (int i = 0; i < 16; ++i) {
                                o0[i] += f * ol0[i];
                                o1[i] += f * ol1[i];
                            }
                        }
                    }
                }
            } else {
                for (int ct = 0; ct < (GEOM == GEOM_2DP ? 2 : 1) * g.nctile; ++ct) {
                    FMA_NEXT_TILE();
                    int ctl = ct;
                    if constexpr (GEOM == GEOM_2DP) {
                        const int c_ = ct >= g.nctile ? 1 : 0;
                        if (c_ != (wave >> 1)) continue;
                        ctl = ct - c_ * g.nctile;
                    }
                    const unsigned long long ml = sm.cmask[cst] >> (4 * hh);
                    const int nsb = nslot - ctl * KT > 32 ? 2 : 1;
#pragma unroll 1
                    for (int sb = 0; sb < nsb; ++sb)
                        block_levels_pv(block_scores(kt + sb * BLK, koff, qb, cneg), vt + sb * BLK, voff,
                                        (uint32_t)(ml >> (32 * sb)), lnear, sgrp, o0, o1);
                }
            }
        } else {
            // (2D pairs: the left cell's coarse tiles, then the right cell's,
            // each taken by its own waves)
            for (int ct = 0; ct < (GEOM == GEOM_2DP ? 2 : 1) * g.nctile; ++ct) {
                FMA_NEXT_TILE();
                int ctl = ct;
                if constexpr (GEOM == GEOM_2DP) {
                    const int c_ = ct >= g.nctile ? 1 : 0;
                    if (c_ != (wave >> 1)) continue;
                    ctl = ct - c_ * g.nctile;
                }
                const unsigned long long ml = sm.cmask[cst] >> (4 * hh);
                const int nsb = nslot - ctl * KT > 32 ? 2 : 1;
#pragma unroll 1
                for (int sb = 0; sb < nsb; ++sb) {
                    attend_block<MASK_SLOTS>(kt + sb * BLK, vt + sb * BLK, koff, voff, qb, 0,
                                             (uint32_t)(ml >> (32 * sb)), first, o0, o1, cneg, mrun, lrun);
                    first = false;
                }
            }
        }

        if constexpr (LIN) {
            // fold the far field in: one source of score M, weight Z and value U / Z
            const float lin_m = lin_u[0], lin_z = lin_u[1];
            if (lin_z > 0.f) {
                const float mnew = fmaxf(mrun, lin_m);
                const float fo = fast_exp2(mrun - mnew), fc = fast_exp2(lin_m - mnew);
                lrun = lrun * fo + (hh == 0 ? lin_z * fc : 0.f);
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int ch = 8 * (i >> 2) + 4 * hh + (i & 3);
                    o0[i] = o0[i] * fo + fc * lin_u[2 + ch];
                    o1[i] = o1[i] * fo + fc * lin_u[2 + 32 + ch];
                }
            }
        }

        // ---------------------------------------- block done: O = O^T / l
        const float inv = 1.0f / sum_pair(lrun);
        const long long qtok = block_token<GEOM>(cb, g, wave * 32 + l32);
        __bf16 *op = outp + ((long long)cb.slice * g.n + qtok) * kHeadDim;
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
            const int d = gq * 8 + 4 * hh;
            *reinterpret_cast<uint2 *>(op + d) =
                make_uint2(pack_bf16(o0[4 * gq] * inv, o0[4 * gq + 1] * inv),
                           pack_bf16(o0[4 * gq + 2] * inv, o0[4 * gq + 3] * inv));
            *reinterpret_cast<uint2 *>(op + 32 + d) =
                make_uint2(pack_bf16(o1[4 * gq] * inv, o1[4 * gq + 1] * inv),
                           pack_bf16(o1[4 * gq + 2] * inv, o1[4 * gq + 3] * inv));
        }
        stored = true;
    }
}

#undef FMA_NEXT_TILE
#undef FMA_ISSUE_NEXT
#undef FMA_ISSUE_SCALAR
#undef FMA_ISSUE_VGPR
#undef FMA_BUILD_LISTS
#undef FMA_SLOT_ENTRY

// FMA-linear far field of every query block, bf16: one wave per block.  The
// block's coarse query of each level scores that level's interaction-list
// rows (one slot per lane, log2 units); M = max over the slots, Z = sum
// 2^(s - M) and U = sum 2^(s - M) v_bar (lane = channel), slots in ascending
// order.  Row: M, Z, U[0 .. 63].  Every coarse-row load is checked against
// the coarse arrays' size.
template <int GEOM>
__global__ __launch_bounds__(64) void lin_far_kernel(AttnArgs a)
{
    constexpr int K = GEOM == GEOM_2D ? kSlots2D : kSlots1D;
    __shared__ float lsc[MAX_SLOTS];
    __shared__ int lrow[MAX_SLOTS];
    const int lane = threadIdx.x;
    const long long id = blockIdx.x;   // slice * tiles_per_slice + block
    const int slice = (int)(id / a.tiles_per_slice);
    const int qt = (int)(id - (long long)slice * a.tiles_per_slice);
    const int cx = GEOM == GEOM_2D ? qt / a.nby : 0, cy = GEOM == GEOM_2D ? qt - (qt / a.nby) * a.nby : 0;
    const int nslot = a.nslot < MAX_SLOTS ? a.nslot : MAX_SLOTS;
    const long long lim = (long long)a.nslice * a.R * kHeadDim;
    const __bf16 *kbg = static_cast<const __bf16 *>(a.kbar), *qbg = static_cast<const __bf16 *>(a.qbar);
    const __bf16 *vbg = static_cast<const __bf16 *>(a.vbar);
    for (int e = lane; e < nslot; e += 64) {
        const int set = e / K, j = e - (e / K) * K;
        float sc = -INFINITY;
        int row = -1;
        if (set < a.lv.nlev) {
            const int lvl = a.lv.lvl[set], M = a.lv.M[set];
            int gi;
            long long gq;
            if constexpr (GEOM == GEOM_2D) {
                gi = list2d_entry(cx, cy, lvl, j, M, a.lv.My[set]);
                gq = (long long)(cx >> (lvl - 1)) * a.lv.My[set] + (cy >> (lvl - 1));
            } else {
                gi = list1d_entry(qt, lvl, j, M, 0);
                gq = qt >> (lvl - 1);
            }
            const long long rk = ((long long)slice * a.R + a.lv.off[set] + gi) * kHeadDim;
            const long long rq = ((long long)slice * a.R + a.lv.off[set] + gq) * kHeadDim;
            if (gi >= 0 && rk >= 0 && rk + kHeadDim <= lim && rq >= 0 && rq + kHeadDim <= lim) {
                const uint4 *kp = reinterpret_cast<const uint4 *>(kbg + rk);
                const uint4 *qp = reinterpret_cast<const uint4 *>(qbg + rq);
                float dot = 0.f;
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    const uint4 kw = kp[c], qw = qp[c];
                    const uint32_t ka[4] = {kw.x, kw.y, kw.z, kw.w}, qa[4] = {qw.x, qw.y, qw.z, qw.w};
#pragma unroll
                    for (int x = 0; x < 4; ++x)
                        dot += bf16lo_to_f32(ka[x]) * bf16lo_to_f32(qa[x]) + bf16hi_to_f32(ka[x]) * bf16hi_to_f32(qa[x]);
                }
                sc = dot * a.scale_log2;
                row = a.lv.off[set] + gi;
            }
        }
        lsc[e] = sc;
        lrow[e] = row;
    }
    __syncthreads();
    float mm = -INFINITY;
    for (int e = lane; e < nslot; e += 64) mm = fmaxf(mm, lsc[e]);
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1) mm = fmaxf(mm, __shfl_xor(mm, sh));
    // Z and U in slot order.  Eight slots at a time, with unconditional loads
    // so that all eight are in flight together: a slot without a row reads
    // element `lane` instead, which is in bounds here because some slot held
    // a full row (mm is finite), and its weight is exactly 0.
    float z = 0.f, u = 0.f;
    if (mm > -INFINITY) {
        for (int e0 = 0; e0 < nslot; e0 += 8) {
            float pv[8], vv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int e = e0 + j;
                const int ec = e < nslot ? e : nslot - 1;
                const int row = e < nslot ? lrow[ec] : -1;
                const long long rv = ((long long)slice * a.R + row) * kHeadDim + lane;
                const bool ok = row >= 0 && rv < lim;
                const float v = static_cast<float>(vbg[ok ? rv : (long long)lane]);
                pv[j] = row >= 0 ? fast_exp2(lsc[ec] - mm) : 0.f;
                vv[j] = ok ? v : 0.f;
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                z += pv[j];
                u += pv[j] * vv[j];
            }
        }
    }
    const long long base = id * (kHeadDim + 2);
    if (base + kHeadDim + 2 <= a.lin_far_elems) {
        a.lin_far[base + 2 + lane] = u;
        if (lane == 0) {
            a.lin_far[base] = mm;
            a.lin_far[base + 1] = z;
        }
    }
}

// Resident workgroups of one kernel variant on the current device (one per
// CU slot).
template <int NW, int GEOM, bool PL, bool LIN>
int resident_groups()
{
    return resident_slots(reinterpret_cast<const void *>(&attend_mfma_kernel<NW, GEOM, PL, LIN>), 64 * NW, 0);
}

// Workgroups per resident slot.  Workgroups that share a CU progress at
// unequal rates (a grid of one workgroup per slot, 16 blocks each at 1D
// 65536 x 128, ended between 62 % and 100 % of the kernel's time), so the
// grid holds several short ranges per slot and the hardware dispatcher
// hands the slots that free up early the ranges not yet started.  More
// workgroups cost one set-up (set table, first tiles) each: four per slot
// measured best in 1D, eight on 2D maps.
template <int GEOM>
constexpr int kGroupsPerSlot = kIs2D<GEOM> ? 8 : 4;

template <int NW, int GEOM, bool PL, bool LIN>
hipError_t launch_nw(const AttnArgs &a, hipStream_t st)
{
    const long long blocks = (long long)(GEOM == GEOM_2DP ? a.tiles_per_slice / 2 : a.tiles_per_slice) * a.nslice;
    const int slots = resident_groups<NW, GEOM, PL, LIN>();
    if (slots <= 0) return hipErrorInvalidDevice;
    const long long want = (long long)slots * kGroupsPerSlot<GEOM>;
    const unsigned grid = (unsigned)(blocks < want ? blocks : want);
    hipLaunchKernelGGL((attend_mfma_kernel<NW, GEOM, PL, LIN>), dim3(grid), dim3(64 * NW), 0, st, a);
    return hipGetLastError();
}

template <int GEOM, bool PL, bool LIN = false>
hipError_t launch_geom(const AttnArgs &a, hipStream_t st)
{
    switch (a.qtile / 32) {
    case 2: return launch_nw<2, GEOM, PL, LIN>(a, st);
    case 4: return launch_nw<4, GEOM, PL, LIN>(a, st);
    case 6: return launch_nw<6, GEOM, PL, LIN>(a, st);
    case 8: return launch_nw<8, GEOM, PL, LIN>(a, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_lin_far(const AttnArgs &a, int geometry, hipStream_t st)
{
    const long long nb = (long long)a.nslice * a.tiles_per_slice;
    if (nb == 0 || a.lv.nlev == 0) return hipSuccess;
    if (nb * (kHeadDim + 2) > a.lin_far_elems || nb >= (1LL << 31)) return hipErrorInvalidValue;
    if (geometry == GEOM_2D)
        hipLaunchKernelGGL(lin_far_kernel<GEOM_2D>, dim3((unsigned)nb), dim3(64), 0, st, a);
    else
        hipLaunchKernelGGL(lin_far_kernel<GEOM_1D>, dim3((unsigned)nb), dim3(64), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_attend_bf16(const AttnArgs &a, int geometry, hipStream_t st)
{
    if (a.nslice == 0 || a.tiles_per_slice == 0) return hipSuccess;
    if (a.nslot > MAX_SLOTS) return hipErrorInvalidValue;
    if (a.qbar && a.nslot > 0) {   // FMA-linear (joint normalisation, rank 1)
        if (a.norm_level || a.rank != 1) return hipErrorInvalidValue;
        if (geometry == GEOM_1D) return launch_geom<GEOM_1D, false, true>(a, st);
        if (geometry == GEOM_2D) return launch_geom<GEOM_2D, false, true>(a, st);
        return hipErrorInvalidValue;
    }
    if (a.norm_level && a.nslot > 0) {   // printed per-level normalisation
        if (geometry == GEOM_1D) return launch_geom<GEOM_1D, true>(a, st);
        if (geometry == GEOM_2D) {
            if (pair_cells_2d(a.r, a.nby, a.nslot, a.norm_level, 0, 1)) return launch_nw<4, GEOM_2DP, true, false>(a, st);
            return launch_geom<GEOM_2D, true>(a, st);
        }
        return hipErrorInvalidValue;
    }
    if (geometry == GEOM_1D) return launch_geom<GEOM_1D, false>(a, st);
    if (geometry == GEOM_2D) {
        if (pair_cells_2d(a.r, a.nby, a.nslot, a.norm_level, 0, 1)) return launch_nw<4, GEOM_2DP, false, false>(a, st);
        return launch_geom<GEOM_2D, false>(a, st);
    }
    return launch_geom<GEOM_DENSE, false>(a, st);
}

}  // namespace fma_dev
