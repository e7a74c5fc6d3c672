// backward.hip -- gradients of the FMA forward pass on gfx950 (end-to-end
// training of the aggregation weights, Sec. 3).
//
// For a loss with upstream gradient dO, per query i and source t (near token
// or coarse row of its interaction list):
//     P_it = exp2(c s_it - lse_i)          c = tau log2(e), lse_i in log2 units
//     dS_it = P_it (dO_i . v_t - D_i)       D_i = dO_i . O_i
// Under the printed per-level normalisation (Eq. fma1d / fma2d as printed)
// the near field and every level are softmax groups of their own, and O is
// the sum of the groups' averages O_G: lse and D are then per group, with
// D_G = dO_i . O_G.  The query pass takes the coarse tiles first (a level's
// slots lie in one aligned group of a 32-slot block, so each level's softmax
// and D_G come out of one block), and the near field's D_N = D - sum_G D_G;
// the key pass sees the near field's lse and D_N.
// FMA-linear (reading R18): a query scores its coarse slots with the coarse
// query of its own group (the same for every query of a base block), so the
// slots' score gradients go to the coarse queries: with c_g = sum over the
// block's queries of dS_ig, dK_bar_g += tau c_g q_bar and dQ_bar += tau c_g
// k_bar_g; dq of a token is its near-field part plus pi^q * dQ_bar of its
// groups (bwd_qreduce, bwd_qapply), and dpi^q comes from q_t . dQ_bar as
// dpi^k does from k_t . dK_bar.
//     dq_i = tau sum_t dS_it k_t,  dk_t += tau dS_it q_i,  dv_t += P_it dO_i
// and the coarsening is linear, so a coarse row's gradient flows back as
//     dk_j += pi[j - start] dk_bar,   dpi[o] += k_(start+o) . dk_bar.
//
// Kernels, in launch order (the forward's coarsening rebuilds K_bar, V_bar):
//   bwd_query   a wave per 32 queries (waves of one block share the tiles):
//               D_i = rowsum(dO * O) of its queries (written for bwd_key); one
//               pass over the query's tiles for lse and dQ (online rescaling
//               against a reference maximum raised only when the weights
//               would overflow, as in the forward), then a pass over its
//               coarse tiles, where the scores with the slots on the lanes
//               give each wave's part of dK_bar, dV_bar (Q^T dS, dO^T P) per
//               slot; the workgroup adds its waves' parts (two-wave groups:
//               one channel half each over both waves' queries) and stores
//               one partial row
//   bwd_reduce  each coarse row adds the partial rows of the workgroups whose
//               lists hold it, in a fixed order (the inverse of the closed-form
//               lists), eight partial rows in flight per wave
//   bwd_key     a wave per 32 keys (waves of one block share the tiles): the
//               query tiles of the key's near window give dK, dV; the epilogue
//               adds pi * dK_bar of every coarse set and writes k_t . dK_bar
//               for the weight gradients (bf16: both on the matrix cores)
//   bwd_row_lines, bwd_col_lines
//               (2D) sum the dot products along pixel rows and columns
//   bwd_weights sums those dot products (2D: line sums) into dpi^k, dpi^v
//               (1D: bwd_weights1d, a workgroup per 64 entries of a set with
//               many terms per entry, bwd_weights1d_narrow a thread per entry)
// No atomics: every sum has a fixed order, so results are reproducible.
//
// Matrix cores: v_mfma_f32_32x32x16_bf16 (bf16 I/O) or v_mfma_f32_32x32x2f32
// (fp32 I/O), fp32 accumulation.  In a 32x32 accumulator lane L holds column
// L & 31 and rows 8 (i >> 2) + 4 (L >> 5) + (i & 3), i < 16; a contraction
// over those rows takes them as the B operand and reads the A operand from a
// transposed LDS copy in the same row order.
//
// Every global load and store is checked against the size of its buffer
// (elements, from the argument block); out-of-range loads read 0 and
// out-of-range stores are dropped.
#include "fma_device.hpp"
#include "fma_kernels.hpp"

namespace fma_dev {

namespace {

constexpr int KT = 64;     // rows per tile
constexpr int PB = 72;     // LDS pitch (bf16 elements) of 64-entry rows
constexpr int PF = 68;     // LDS pitch (fp32 elements) of 64-entry rows
constexpr int PQB = 40;    // LDS pitch (bf16) of 32-entry transposed rows
constexpr int PQF = 36;    // LDS pitch (fp32) of 32-entry transposed rows
constexpr int kMaxSlots = 448;   // interaction-list slots a plan may have

template <bool BF16>
struct Elt;
template <>
struct Elt<true> {
    typedef __bf16 T;
    static constexpr int P = PB, PQ = PQB, PER16 = 8;   // elements per 16-byte chunk
};
template <>
struct Elt<false> {
    typedef float T;
    static constexpr int P = PF, PQ = PQF, PER16 = 4;
};

// ------------------------------------------------------------- checked memory
__device__ inline uint4 ld16(const void *base, long long elem, int esize, long long lim)
{
    // 16 bytes starting at element `elem` (a multiple of 16 / esize)
    if (elem < 0 || elem + 16 / esize > lim) return make_uint4(0, 0, 0, 0);
    return *reinterpret_cast<const uint4 *>(static_cast<const char *>(base) + elem * esize);
}

__device__ inline float ldf(const float *p, long long i, long long lim) { return (i >= 0 && i < lim) ? p[i] : 0.f; }

__device__ inline void stf(float *p, long long i, long long lim, float x)
{
    if (i >= 0 && i < lim) p[i] = x;
}

__device__ inline void st4f(float *p, long long i, long long lim, float a, float b, float c, float d)
{
    if (i >= 0 && i + 4 <= lim) *reinterpret_cast<float4 *>(p + i) = make_float4(a, b, c, d);
}

// 4 consecutive output elements of the I/O dtype
template <bool BF16>
__device__ inline void st4(void *base, long long i, long long lim, float a, float b, float c, float d)
{
    if (i < 0 || i + 4 > lim) return;
    if constexpr (BF16)
        *reinterpret_cast<uint2 *>(static_cast<__bf16 *>(base) + i) = make_uint2(pack_bf16x2(a, b), pack_bf16x2(c, d));
    else
        *reinterpret_cast<float4 *>(static_cast<float *>(base) + i) = make_float4(a, b, c, d);
}

__device__ inline float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ inline int acc_row(int i, int hh) { return 8 * (i >> 2) + 4 * hh + (i & 3); }

// ------------------------------------------------------------- operands
// A row operand: this lane's part of one 64-channel row (lane & 31 = row,
// lane >> 5 = which channels), as the A or the B side of a 32x32 MFMA.
template <bool BF16>
struct RowOp;
template <>
struct RowOp<true> {
    bf16x8 x[4];   // channels 16 c + 8 hh .. + 7
    __device__ void from_lds(const __bf16 *row, int hh)
    {
#pragma unroll
        for (int c = 0; c < 4; ++c) x[c] = *reinterpret_cast<const bf16x8 *>(row + 16 * c + 8 * hh);
    }
    __device__ float chan(int c, int e) const { return static_cast<float>(x[c][e]); }
};
template <>
struct RowOp<false> {
    float x[32];   // channel 2 c + hh
    __device__ void from_lds(const float *row, int hh)
    {
#pragma unroll
        for (int c = 0; c < 32; ++c) x[c] = row[2 * c + hh];
    }
};

// acc[m][n] += sum over the 64 channels of A[m][ch] B[n][ch]
template <bool BF16>
__device__ inline f32x16 contract_channels(const RowOp<BF16> &A, const RowOp<BF16> &B, f32x16 acc)
{
    if constexpr (BF16) {
#pragma unroll
        for (int c = 0; c < 4; ++c) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A.x[c], B.x[c], acc, 0, 0, 0);
    } else {
#pragma unroll
        for (int c = 0; c < 32; ++c) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(A.x[c], B.x[c], acc, 0, 0, 0);
    }
    return acc;
}

// out_db[ch][n] += sum over 32 rows r of T[ch][rowbase + r] w[r][n], for
// ch = 32 db + (lane & 31); w in accumulator layout (column n = lane & 31).
template <bool BF16>
__device__ inline void contract_rows(const typename Elt<BF16>::T *T, int pitch, int rowbase, const f32x16 &w, int l32,
                                     int hh, f32x16 &out0, f32x16 &out1)
{
    if constexpr (BF16) {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            bf16x8 pb;
#pragma unroll
            for (int e = 0; e < 8; ++e) pb[e] = static_cast<__bf16>(w[8 * hf + e]);
            const int base = rowbase + 16 * hf + 4 * hh;
#pragma unroll
            for (int db = 0; db < 2; ++db) {
                const __bf16 *t = T + (db * 32 + l32) * pitch + base;
                const bf16x4 lo = *reinterpret_cast<const bf16x4 *>(t);
                const bf16x4 hi = *reinterpret_cast<const bf16x4 *>(t + 8);
                const bf16x8 av = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                if (db == 0)
                    out0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb, out0, 0, 0, 0);
                else
                    out1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb, out1, 0, 0, 0);
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int row = rowbase + acc_row(i, hh);
            out0 = __builtin_amdgcn_mfma_f32_32x32x2f32(T[l32 * pitch + row], w[i], out0, 0, 0, 0);
            out1 = __builtin_amdgcn_mfma_f32_32x32x2f32(T[(32 + l32) * pitch + row], w[i], out1, 0, 0, 0);
        }
    }
}

// bf16 tiles in LDS: 64-channel rows of 128 bytes whose 16-byte chunk c sits
// at chunk c ^ swz(row).  For the row reads of a 32x32 operand (ds_read_b128,
// lane = row) the rows of any 16 lanes land in distinct bank groups, and for
// the transposing reads (ds_read_b64_tr_b16, four rows of four chunks per 16
// lanes) rows r and r + 2 sit in opposite 64-byte halves, so neither kind
// conflicts; fp32 tiles keep the padded pitch.
__device__ inline int swz(int row) { return (2 * (row & 3)) ^ ((row >> 2) & 1) ^ (2 * ((row >> 3) & 1)); }
__device__ inline int sw_off(int row, int chunk) { return row * kHeadDim + 8 * (chunk ^ swz(row)); }

// this lane's part of row `row` of a swizzled bf16 tile (as RowOp::from_lds)
__device__ inline void row_from_tile(RowOp<true> &op, const __bf16 *tile, int row, int hh)
{
#pragma unroll
    for (int c = 0; c < 4; ++c) op.x[c] = *reinterpret_cast<const bf16x8 *>(tile + sw_off(row, 2 * c + hh));
}

// contract_rows on a swizzled bf16 tile read with transposing loads: the A
// operand of lane (l32, hh) is channel 32 db + l32 at rows rowbase + 16 hf +
// {4 hh .. 4 hh + 3, 8 + 4 hh .. 8 + 4 hh + 3}, the order of the B operand's
// k slots.  Lanes 16 g + 4 j + q read rows 4 (g >> 1) + j (and + 8), chunk
// 4 db + 2 (g & 1) + (q >> 1), half q & 1.
__device__ inline void contract_rows_tr(const __bf16 *tile, int rowbase, const f32x16 &w, int lane, f32x16 &out0,
                                        f32x16 &out1)
{
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const int gq = lane >> 4, s4 = lane & 15, j = s4 >> 2, q = s4 & 3;
    const int row = 4 * (gq >> 1) + j;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
        bf16x8 pb;
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[e] = static_cast<__bf16>(w[8 * hf + e]);
        const __bf16 *t16 = tile + (rowbase + 16 * hf) * kHeadDim;
#pragma unroll
        for (int db = 0; db < 2; ++db) {
            const int chunk = 4 * db + 2 * (gq & 1) + (q >> 1);
            const s16x4 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_s16x4 *)(t16 + sw_off(row, chunk) + 4 * (q & 1)));
            const s16x4 r2 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_s16x4 *)(t16 + sw_off(row + 8, chunk) + 4 * (q & 1)));
            typedef short s16x8 __attribute__((ext_vector_type(8)));
            const s16x8 av = {r1[0], r1[1], r1[2], r1[3], r2[0], r2[1], r2[2], r2[3]};
            const bf16x8 va = __builtin_bit_cast(bf16x8, av);
            if (db == 0)
                out0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, out0, 0, 0, 0);
            else
                out1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, out1, 0, 0, 0);
        }
    }
}

// One channel half db of contract_rows_tr (rows 0..31 of the tile), with the
// B operand given as bf16: pb[hf] holds w's entries 8 hf .. 8 hf + 7.
__device__ inline f32x16 contract_rows_tr1(const __bf16 *tile, const bf16x8 pb[2], int lane, int db, f32x16 out)
{
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const int gq = lane >> 4, s4 = lane & 15, j = s4 >> 2, q = s4 & 3;
    const int row = 4 * (gq >> 1) + j;
    const int chunk = 4 * db + 2 * (gq & 1) + (q >> 1);
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
        const __bf16 *t16 = tile + (16 * hf) * kHeadDim;
        const s16x4 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(t16 + sw_off(row, chunk) + 4 * (q & 1)));
        const s16x4 r2 =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(t16 + sw_off(row + 8, chunk) + 4 * (q & 1)));
        const s16x8 av = {r1[0], r1[1], r1[2], r1[3], r2[0], r2[1], r2[2], r2[3]};
        out = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, av), pb[hf], out, 0, 0, 0);
    }
    return out;
}

// max / sum of x over this lane and lane ^ 32 (v_permlane32_swap: a VALU
// exchange of the wave's halves, no LDS round trip)
__device__ inline float pmax(float x)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float psum(float x)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Per-level softmax of one 32-slot block of scores (per-level
// normalisation): the slots form aligned groups of grp (4, 8, 16 or 32)
// rows, one level each.  x holds the lane's scaled scores (log2 units, -inf
// for empty slots) in accumulator layout (element i is row acc_row(i, hh)),
// so a group of 4 is one chunk of 4 elements, 8 that chunk in both halves of
// the wave (lane ^ 32), 16 two chunks and 32 all four.  On return x holds
// dS = P (dP - D_g) with P = exp2(x - m_g) / l_g; lse[c] = m_g + log2 l_g
// (-inf for an empty group) and dg[c] = D_g = sum_g P dP of the group of
// chunk c.
__device__ inline void level_block(f32x16 &x, const f32x16 &dp, int grp, float (&lse)[4], float (&dg)[4])
{
    float cm[4], cl[4], cd[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) cm[c] = fmaxf(fmaxf(x[4 * c], x[4 * c + 1]), fmaxf(x[4 * c + 2], x[4 * c + 3]));
    if (grp >= 16) {
        cm[0] = cm[1] = fmaxf(cm[0], cm[1]);
        cm[2] = cm[3] = fmaxf(cm[2], cm[3]);
    }
    if (grp >= 32) cm[0] = cm[1] = cm[2] = cm[3] = fmaxf(cm[0], cm[2]);
    if (grp >= 8) {
#pragma unroll
        for (int c = 0; c < 4; ++c) cm[c] = pmax(cm[c]);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        cm[c] = cm[c] > -INFINITY ? cm[c] : 0.0f;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[4 * c + e] = fexp2(x[4 * c + e] - cm[c]);
        cl[c] = (x[4 * c] + x[4 * c + 1]) + (x[4 * c + 2] + x[4 * c + 3]);
    }
    if (grp >= 16) {
        cl[0] = cl[1] = cl[0] + cl[1];
        cl[2] = cl[3] = cl[2] + cl[3];
    }
    if (grp >= 32) cl[0] = cl[1] = cl[2] = cl[3] = cl[0] + cl[2];
    if (grp >= 8) {
#pragma unroll
        for (int c = 0; c < 4; ++c) cl[c] = psum(cl[c]);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const float inv = cl[c] > 0.0f ? 1.0f / cl[c] : 0.0f;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[4 * c + e] *= inv;
        cd[c] = (x[4 * c] * dp[4 * c] + x[4 * c + 1] * dp[4 * c + 1]) +
                (x[4 * c + 2] * dp[4 * c + 2] + x[4 * c + 3] * dp[4 * c + 3]);
    }
    if (grp >= 16) {
        cd[0] = cd[1] = cd[0] + cd[1];
        cd[2] = cd[3] = cd[2] + cd[3];
    }
    if (grp >= 32) cd[0] = cd[1] = cd[2] = cd[3] = cd[0] + cd[2];
    if (grp >= 8) {
#pragma unroll
        for (int c = 0; c < 4; ++c) cd[c] = psum(cd[c]);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[4 * c + e] *= dp[4 * c + e] - cd[c];
        lse[c] = cl[c] > 0.0f ? cm[c] + __log2f(cl[c]) : -INFINITY;
        dg[c] = cd[c];
    }
}

// token of position p (0 .. qtile-1) of block b
template <bool TWO_D>
__device__ inline long long block_tok(const BwdArgs &a, int b, int p)
{
    if constexpr (TWO_D) {
        const int cx = b / a.nby, cy = b - (b / a.nby) * a.nby;
        return (long long)(cx * a.r + p / a.r) * a.side + cy * a.r + p % a.r;
    } else {
        return (long long)b * a.r + p;
    }
}

// --------------------------------------------------------------- tiles
// 2D: the in-map 3x3 neighbourhood of a cell is a rectangle of cells, walked
// row-major (the forward's order); near cell ci is cell (x0 + ci / ny,
// y0 + ci % ny).
struct Near2D {
    int x0, y0, ny, ncell;
};

__device__ inline Near2D near2d(const BwdArgs &a, int b)
{
    const int cx = b / a.nby, cy = b - (b / a.nby) * a.nby;
    Near2D d;
    d.x0 = cx > 0 ? cx - 1 : 0;
    d.y0 = cy > 0 ? cy - 1 : 0;
    const int x1 = cx + 1 < a.nbx ? cx + 1 : cx, y1 = cy + 1 < a.nby ? cy + 1 : cy;
    d.ny = y1 - d.y0 + 1;
    d.ncell = (x1 - d.x0 + 1) * d.ny;
    return d;
}

// token of position p (row-major in the r x r cell, lg = log2 r) of near cell ci
__device__ inline long long near2d_token(const BwdArgs &a, const Near2D &d, int ci, int p, int lg)
{
    const int qx = ci / d.ny;
    const int ux = d.x0 + qx, uy = d.y0 + ci - qx * d.ny;
    return (long long)((ux << lg) + (p >> lg)) * a.side + (uy << lg) + (p & (a.r - 1));
}

// Coarse row of interaction-list slot `slot` of block b, or -1 for an empty
// slot.  Joint layout: slot = set * K + j; per-level layout: slot = level *
// slot_group + basis * K + j (slots past a level's rank * K are padding).
template <bool TWO_D>
__device__ inline int coarse_source(const BwdArgs &a, int b, int slot)
{
    constexpr int K = TWO_D ? kSlots2D : kSlots1D;
    if (slot >= a.nslot) return -1;
    int set, j;
    if (a.norm_level) {
        const int lev = slot / a.slot_group, rem = slot - lev * a.slot_group;
        const int basis = rem / K;
        if (basis >= a.rank) return -1;
        set = lev * a.rank + basis;
        j = rem - basis * K;
    } else {
        set = slot / K;
        j = slot - set * K;
    }
    if (set >= a.lv.nlev) return -1;
    int g;
    if constexpr (TWO_D)
        g = list2d_entry(b / a.nby, b % a.nby, a.lv.lvl[set], j, a.lv.M[set], a.lv.My[set]);
    else
        g = list1d_entry(b, a.lv.lvl[set], j, a.lv.M[set], a.causal);
    return g < 0 ? -1 : a.lv.off[set] + g;
}

// The key tiles of one query block, in the forward's order: near tiles (1D:
// blocks b-1 .. b+1, causal b-1 .. b; 2D: the in-map 3x3 cells, r*r/64 tiles
// each), then the interaction-list slots, 64 per tile, whose coarse rows
// come from a table built once per workgroup (csrc, in LDS).  Blocks smaller
// than a tile (1D r = 16, 32; 2D 4 x 4 cells) pack the near field's tokens
// 64 to a tile, cell after cell, and the rows past it are empty (full =
// false: the near tiles' rows are masked by their validity flags).
struct QTiles {
    int nnear, ntile, tpc, lg;
    long long klo;        // 1D: first near key
    long long khi;        // 1D: one past the last near key
    int csz;              // 2D: tokens per cell
    bool full;            // every near-tile row is a near token
    Near2D nd;            // 2D: near cells
    const int *csrc;      // coarse row of every slot (-1: empty)
};

template <bool TWO_D>
__device__ inline QTiles query_tiles(const BwdArgs &a, int b, const int *csrc)
{
    QTiles m;
    m.klo = 0;
    m.tpc = 1;
    m.lg = 31 - __builtin_clz(a.r);
    m.csrc = csrc;
    m.nd = Near2D{0, 0, 1, 0};
    m.khi = 0;
    m.csz = 1;
    if constexpr (TWO_D) {
        m.csz = a.qtile;
        m.tpc = a.qtile / KT;
        m.nd = near2d(a, b);
        m.nnear = (m.nd.ncell * m.csz + KT - 1) / KT;
        m.full = m.csz % KT == 0;
    } else {
        const long long lo = b > 0 ? (long long)(b - 1) * a.r : 0;
        long long hi = a.causal ? (long long)(b + 1) * a.r : (long long)(b + 2) * a.r;
        if (hi > a.n) hi = a.n;
        m.klo = lo;
        m.khi = hi;
        m.nnear = (int)((hi - lo + KT - 1) / KT);
        m.full = (hi - lo) % KT == 0;
    }
    m.ntile = m.nnear + (a.nslot + KT - 1) / KT;
    return m;
}

// One 64-row K (and V) tile in registers: NT threads, 16 bytes each per
// load (near rows from the tile's geometry, coarse rows from the slot
// table); stash() writes it to LDS (K and V row-major,
// K also transposed) and the row validity flags.
template <bool BF16, bool TWO_D, int NT, bool WITH_V>
struct KVTile {
    typedef typename Elt<BF16>::T T;
    static constexpr int PER = Elt<BF16>::PER16, CPR = kHeadDim / PER, P = Elt<BF16>::P;
    static constexpr int ITER = KT * CPR / NT;
    static_assert(KT * CPR % NT == 0, "tile split");
    uint4 kr[ITER], vr[WITH_V ? ITER : 1];
    int ok[ITER];

    __device__ void fetch(const BwdArgs &a, const QTiles &m, int b, int t, int slice, int tid)
    {
        constexpr int ES = BF16 ? 2 : 4;
        // the tile's uniform part once: near rows are base + row (1D) or
        // pixel pofs + row of a cell starting at token base (2D); coarse rows
        // come from the slot table
        const bool co = t >= m.nnear;
        long long base = 0;
        int pofs = 0;
        if (!co) {
            if constexpr (TWO_D) {
                if (m.full) {
                    const int ci = t / m.tpc;
                    pofs = (t - ci * m.tpc) * KT;
                    base = near2d_token(a, m.nd, ci, 0, m.lg);
                }
            } else {
                base = m.klo + (long long)t * KT;
            }
        }
        const int slot0 = (t - m.nnear) * KT;
#pragma unroll
        for (int it = 0; it < ITER; ++it) {
            const int c = tid + it * NT;
            const int row = c / CPR, col = c - (c / CPR) * CPR;
            long long src;
            if (co) {
                const int slot = slot0 + row;
                src = slot < a.nslot && slot < kMaxSlots ? m.csrc[slot] : -1;
            } else if constexpr (TWO_D) {
                if (m.full) {
                    const int p = pofs + row;
                    src = base + (long long)(p >> m.lg) * a.side + (p & (a.r - 1));
                } else {
                    // packed cells: position t * 64 + row of the near tokens
                    const int pg = t * KT + row;
                    const int ci = pg / m.csz;
                    src = ci < m.nd.ncell ? near2d_token(a, m.nd, ci, pg - ci * m.csz, m.lg) : -1;
                }
            } else {
                src = base + row;
                if (src >= m.khi) src = -1;
            }
            kr[it] = make_uint4(0, 0, 0, 0);
            if constexpr (WITH_V) vr[it] = make_uint4(0, 0, 0, 0);
            ok[it] = src >= 0;
            if (src >= 0) {
                const long long e = co ? ((long long)slice * a.R + src) * kHeadDim + col * PER
                                       : ((long long)slice * a.n + src) * kHeadDim + col * PER;
                kr[it] = ld16(co ? a.kbar : a.k, e, ES, co ? a.coarse_elems : a.io_elems);
                if constexpr (WITH_V) vr[it] = ld16(co ? a.vbar : a.v, e, ES, co ? a.coarse_elems : a.io_elems);
            }
        }
    }

    // bf16: swizzled rows (the transposed operand comes from transposing
    // reads); fp32: padded rows plus a transposed copy of K
    __device__ void stash(T *sk, T *skt, T *sv, int *valid, int tid) const
    {
#pragma unroll
        for (int it = 0; it < ITER; ++it) {
            const int c = tid + it * NT;
            const int row = c / CPR, col = c - (c / CPR) * CPR;
            const int o = BF16 ? sw_off(row, col) : row * P + col * PER;
            *reinterpret_cast<uint4 *>(sk + o) = kr[it];
            if (col == 0) valid[row] = ok[it];
            if constexpr (WITH_V) {
                *reinterpret_cast<uint4 *>(sv + o) = vr[it];
                if constexpr (!BF16) {
                    const T *kv = reinterpret_cast<const T *>(&kr[it]);
#pragma unroll
                    for (int e = 0; e < PER; ++e) skt[(col * PER + e) * P + row] = kv[e];
                }
            }
        }
    }
};

// --------------------------------------------------------------- bwd_query
template <bool BF16, int NW, bool PL, bool LIN>
struct QSmem {
    typedef typename Elt<BF16>::T T;
    T k[BF16 ? KT * kHeadDim : KT * Elt<BF16>::P];
    T kt[BF16 ? 8 : kHeadDim * Elt<BF16>::P];   // fp32 only: K transposed
    T v[BF16 ? KT * kHeadDim : KT * Elt<BF16>::P];
    // Q and dO of each wave's 32 queries: bf16 as swizzled rows (transposing
    // reads give Q^T, dO^T), fp32 transposed
    T qt[NW][BF16 ? 32 * kHeadDim : kHeadDim * Elt<BF16>::PQ];
    T dot[NW][BF16 ? 32 * kHeadDim : kHeadDim * Elt<BF16>::PQ];
    __attribute__((aligned(16))) int valid[KT];   // read four rows at a time
    __attribute__((aligned(16))) float lse[NW][32];
    __attribute__((aligned(16))) float dd[NW][32];
    // per-level normalisation: lse and D of every (level, query) of each wave
    __attribute__((aligned(16))) float lsel[PL ? NW : 1][PL ? kMaxCoarse : 1][32];
    __attribute__((aligned(16))) float ddl[PL ? NW : 1][PL ? kMaxCoarse : 1][32];
    // FMA-linear: the block's coarse query of every set, the current coarse
    // tile's slot scores, the waves' slot sums c of one 32-slot block, and
    // the workgroup's dQ_bar of every set
    float qbl[LIN ? kMaxCoarse : 1][LIN ? kHeadDim : 1];
    float lins[LIN ? KT : 1];
    float cw[LIN ? NW : 1][32];
    float dqb[LIN ? kMaxCoarse : 1][LIN ? kHeadDim : 1];
    int csrc[kMaxSlots];   // coarse row of every interaction-list slot of the block
    // the waves' running sum of a coarse partial, [slot][channels]: whole
    // rows (64 channels) for four or more waves, half rows for two, whose
    // workgroups need the smaller LDS to fit four per CU
    __attribute__((aligned(16))) float cred[32 * (NW >= 4 ? 68 : 36)];
};

// One workgroup = NW waves of one query block, wave w taking the block's
// 32-query chunk g * NW + w (g = the workgroup's group within the block;
// waves past the block's chunks only help to load).  The tiles are loaded
// once for all waves, the next one into registers while the current one is
// multiplied out of LDS.
// bf16: registers for two waves per SIMD (1D two-wave groups and the fp32
// operands do not fit without spilling)
template <bool BF16, bool TWO_D, int NW, bool PL, bool LIN>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(BF16 && (TWO_D || NW >= 4) ? 2 : 1))) void bwd_query(BwdArgs a)
{
    static_assert(!(PL && LIN), "FMA-linear uses the joint normalisation");
    constexpr int NT = 64 * NW;
    constexpr int ES = BF16 ? 2 : 4;
    constexpr int PQ = Elt<BF16>::PQ, P = Elt<BF16>::P;
    constexpr int K = TWO_D ? kSlots2D : kSlots1D;
    __shared__ __attribute__((aligned(16))) QSmem<BF16, NW, PL, LIN> sm;
    const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hh = lane >> 5;
    const int wave = tid >> 6;
    const int cpb = (a.qtile + 31) / 32;          // chunks per block
    const int gpb = (cpb + NW - 1) / NW;          // workgroups per block
    const long long wg = blockIdx.x;
    const int ls = (int)(wg / ((long long)a.nblocks * gpb));   // slice within the pass
    const long long rem = wg - (long long)ls * a.nblocks * gpb;
    const int b = (int)(rem / gpb), gi = (int)(rem - (rem / gpb) * gpb);
    const int slice = a.slice0 + ls;
    if (ls >= a.pslices || slice >= a.nslice) return;
    const int cw = gi * NW + wave;                 // this wave's chunk in the block
    const bool active = cw < cpb;
    // lanes past a block smaller than the wave repeat one of its queries with
    // a zero upstream gradient (no contribution) and store nothing
    const bool qlive = active && cw * 32 + l32 < a.qtile;
    for (int sl = tid; sl < a.nslot && sl < kMaxSlots; sl += NT) sm.csrc[sl] = coarse_source<TWO_D>(a, b, sl);
    if constexpr (LIN) {
        // the block's coarse query of every set (rank 1: set = level), and
        // zeroed dQ_bar accumulators
        for (int x = tid; x < kMaxCoarse * kHeadDim; x += NT) {
            const int e = x / kHeadDim, ch = x - (x / kHeadDim) * kHeadDim;
            float val = 0.f;
            if (e < a.lv.nlev) {
                const int sh = a.lv.lvl[e] - 1;
                long long g;
                if constexpr (TWO_D)
                    g = (long long)((b / a.nby) >> sh) * a.lv.My[e] + ((b - (b / a.nby) * a.nby) >> sh);
                else
                    g = b >> sh;
                const long long el = ((long long)slice * a.R + a.lv.off[e] + g) * kHeadDim + ch;
                if (el >= 0 && el < a.coarse_elems) {
                    if constexpr (BF16)
                        val = static_cast<float>(static_cast<const __bf16 *>(a.qbar)[el]);
                    else
                        val = static_cast<const float *>(a.qbar)[el];
                }
            }
            sm.qbl[e][ch] = val;
            sm.dqb[e][ch] = 0.f;
        }
    }
    __syncthreads();
    const QTiles m = query_tiles<TWO_D>(a, b, sm.csrc);
    // FMA-linear: the scores of coarse tile t's slots (one per thread, the
    // block's coarse query of the slot's set against the slot's row), after
    // the tile is in LDS; every thread reaches the barrier
    auto lin_scores = [&](int t) {
        if constexpr (LIN) {
            if (t >= m.nnear && tid < KT) {
                const int slot = (t - m.nnear) * KT + tid;
                float acc = 0.f;
                if (slot < a.nslot && sm.valid[tid]) {
                    int e = slot / K;
                    e = e < kMaxCoarse ? e : kMaxCoarse - 1;
#pragma unroll 8
                    for (int ch = 0; ch < kHeadDim; ++ch) {
                        float kv;
                        if constexpr (BF16)
                            kv = static_cast<float>(sm.k[sw_off(tid, ch >> 3) + (ch & 7)]);
                        else
                            kv = sm.k[tid * P + ch];
                        acc += sm.qbl[e][ch] * kv;
                    }
                }
                sm.lins[tid] = acc;
            }
            __syncthreads();
        }
    };

    // this lane's query: operands of Q and dO (B side), their transposes in LDS
    const long long qtok = active ? block_tok<TWO_D>(a, b, qlive ? cw * 32 + l32 : l32 % a.qtile) : 0;
    const long long qrow = ((long long)slice * a.n + qtok) * kHeadDim;
    // and D = dO . O of the query (this lane's half of the channels, then
    // the other half's from lane ^ 32), written for the key pass
    RowOp<BF16> qo, go;
    float dpart = 0.f;
    if constexpr (BF16) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const uint4 u = ld16(a.q, qrow + 16 * c + 8 * hh, ES, a.io_elems);
            const uint4 g = qlive ? ld16(a.dout, qrow + 16 * c + 8 * hh, ES, a.io_elems) : make_uint4(0, 0, 0, 0);
            const uint4 o = ld16(a.out, qrow + 16 * c + 8 * hh, ES, a.io_elems);
            qo.x[c] = __builtin_bit_cast(bf16x8, u);
            go.x[c] = __builtin_bit_cast(bf16x8, g);
            const bf16x8 ov = __builtin_bit_cast(bf16x8, o);
            *reinterpret_cast<bf16x8 *>(sm.qt[wave] + sw_off(l32, 2 * c + hh)) = qo.x[c];
            *reinterpret_cast<bf16x8 *>(sm.dot[wave] + sw_off(l32, 2 * c + hh)) = go.x[c];
#pragma unroll
            for (int e = 0; e < 8; ++e) dpart += static_cast<float>(go.x[c][e]) * static_cast<float>(ov[e]);
        }
    } else {
        const float *qp = static_cast<const float *>(a.q);
        const float *gp = static_cast<const float *>(a.dout);
        const float *op = static_cast<const float *>(a.out);
#pragma unroll
        for (int c = 0; c < 32; ++c) {
            qo.x[c] = ldf(qp, qrow + 2 * c + hh, a.io_elems);
            go.x[c] = qlive ? ldf(gp, qrow + 2 * c + hh, a.io_elems) : 0.f;
            sm.qt[wave][(2 * c + hh) * PQ + l32] = qo.x[c];
            sm.dot[wave][(2 * c + hh) * PQ + l32] = go.x[c];
            dpart += go.x[c] * ldf(op, qrow + 2 * c + hh, a.io_elems);
        }
    }
    const float dq_row = psum(dpart);
    const float cs = a.scale_log2;
    // 1D: the last query of the workgroup; causal near tiles past it add nothing
    const long long wg_qmax = TWO_D ? 0 : (long long)b * a.r + (long long)(gi * NW + NW) * 32 - 1;
    // number of tiles this workgroup walks (causal: the near tiles up to its queries)
    int tend_near = m.nnear;
    if constexpr (!TWO_D)
        if (a.causal) {
            const long long lim = (wg_qmax - m.klo) / KT + 1;
            tend_near = (int)(lim < m.nnear ? lim : m.nnear);
        }
    const int nco = m.ntile - m.nnear;   // coarse tiles
    const int ntl = tend_near + nco;
    auto tile_of = [&](int x) { return x < tend_near ? x : m.nnear + (x - tend_near); };
    // pass 1 order: the forward's (near tiles, then coarse); per-level: the
    // coarse tiles first, so that the near field's D_N is known before it.
    // Levels wider than a 32-slot block (2D rank p >= 2) walk the coarse
    // tiles twice: a sweep that only forms each level's lse and D_G (online,
    // over the level's blocks), then the sweep that forms dS with them.
    const bool wide = PL && a.slot_group > 32;
    const int nco1 = wide ? 2 * nco : nco;   // coarse steps of pass 1
    const int ntl1 = PL ? tend_near + nco1 : ntl;
    auto tile1 = [&](int x) {
        if constexpr (PL) return x < nco1 ? m.nnear + (x < nco ? x : x - nco) : x - nco1;
        return tile_of(x);
    };

    // ---- pass 1, every tile once: the online max m and sum l of the query's
    // exp2 scores and, with the forward's rescaling, dq = sum_t exp2(s_t - m)
    // (dP_t - D) k_t; dQ = tau dq / l and lse = m + log2 l at the end.  m is
    // raised only when a tile's maximum exceeds it by 2^8 (each query for
    // itself: the other lanes rescale by exp2(0) = 1 exactly).
    float mrun = -1.0e30f, lrun = 0.f;
    f32x16 dq0 = {0}, dq1 = {0};
    // per-level: the coarse slots' part of dq (already normalised), this
    // lane's part of sum_G D_G, and the near field's D_N
    f32x16 dqc0 = {0}, dqc1 = {0};
    float dsum = 0.f, dnear = dq_row;
    // wide levels, stats sweep: the open level's running max, sum of
    // exp2(s - gm) and sum of exp2(s - gm) dP (each query, both lane halves alike)
    float gm = -INFINITY, gl = 0.f, gd = 0.f;
    {
        KVTile<BF16, TWO_D, NT, true> kv;
        if (ntl1 > 0) kv.fetch(a, m, b, tile1(0), slice, tid);
        for (int x = 0; x < ntl1; ++x) {
            const int t = tile1(x);
            const bool near = t < m.nnear;
            const long long key0 = TWO_D ? 0 : m.klo + (long long)t * KT;
            // causal: row kr of the tile is visible iff kr <= qrel (32-bit, clamped)
            const long long qd = qtok - key0;
            const int qrel = qd < -1 ? -1 : qd > KT ? KT : (int)qd;
            __syncthreads();
            kv.stash(sm.k, sm.kt, sm.v, sm.valid, tid);
            __syncthreads();
            lin_scores(t);
            if (x + 1 < ntl1) kv.fetch(a, m, b, tile1(x + 1), slice, tid);
            if (!active) continue;
            if constexpr (PL)
                if (x == nco1) dnear = dq_row - psum(dsum);   // the first near tile
            const bool stats = wide && x < nco;   // wide levels: the stats sweep
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                if (!near && (t - m.nnear) * KT + kb * 32 >= a.nslot) continue;   // past the last slot
                RowOp<BF16> kro, vro;
                if constexpr (BF16) {
                    row_from_tile(kro, sm.k, kb * 32 + l32, hh);
                    row_from_tile(vro, sm.v, kb * 32 + l32, hh);
                } else {
                    kro.from_lds(sm.k + (kb * 32 + l32) * P, hh);
                    vro.from_lds(sm.v + (kb * 32 + l32) * P, hh);
                }
                if constexpr (LIN) {
                    if (!near) {
                        // coarse slots: the block's shared scores; they enter m
                        // and l only (their gradient goes to the coarse queries)
                        f32x16 sc;
                        float mxl = -INFINITY;
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            const int kr = kb * 32 + acc_row(i, hh);
                            sc[i] = sm.valid[kr] != 0 ? sm.lins[kr] * cs : -INFINITY;
                            mxl = fmaxf(mxl, sc[i]);
                        }
                        mxl = pmax(mxl);
                        const bool raise = mxl > mrun + 8.0f;
                        if (__builtin_amdgcn_ballot_w64(raise) != 0) {
                            const float mnew = raise ? mxl : mrun;
                            const float corr = fexp2(mrun - mnew);
                            lrun *= corr;
#pragma unroll
                            for (int i = 0; i < 16; ++i) {
                                dq0[i] *= corr;
                                dq1[i] *= corr;
                            }
                            mrun = mnew;
                        }
#pragma unroll
                        for (int i = 0; i < 16; ++i) lrun += fexp2(sc[i] - mrun);
                        continue;
                    }
                }
                f32x16 s = contract_channels<BF16>(kro, qo, f32x16{0});    // S^T: keys x queries
                f32x16 dp = contract_channels<BF16>(vro, go, f32x16{0});   // dP^T
                if constexpr (PL) {
                    if (!near && wide) {
                        // a level spans whole blocks: its lse and D_G online
                        // over them (stats sweep), then dS = P (dP - D_G) with
                        // P = exp2(s - lse_G) (second sweep)
#pragma unroll
                        for (int i = 0; i < 16; ++i)
                            s[i] = sm.valid[kb * 32 + acc_row(i, hh)] != 0 ? s[i] * cs : -INFINITY;
                        const int sb0 = (t - m.nnear) * KT + kb * 32;   // first slot of the block
                        const int grp = a.slot_group;
                        int lev = sb0 / grp;
                        lev = lev < kMaxCoarse ? lev : kMaxCoarse - 1;
                        if (stats) {
                            if (sb0 % grp == 0) {
                                gm = -INFINITY;
                                gl = 0.f;
                                gd = 0.f;
                            }
                            float bm = -INFINITY;
#pragma unroll
                            for (int i = 0; i < 16; ++i) bm = fmaxf(bm, s[i]);
                            const float mnew = fmaxf(gm, pmax(bm));
                            const float mref = mnew > -INFINITY ? mnew : 0.f;
                            const float corr = gm > -INFINITY ? fexp2(gm - mref) : 0.f;
                            float bl = 0.f, bd = 0.f;
#pragma unroll
                            for (int i = 0; i < 16; ++i) {
                                const float p = fexp2(s[i] - mref);   // 0 for empty slots
                                bl += p;
                                bd += p * dp[i];
                            }
                            gl = gl * corr + psum(bl);
                            gd = gd * corr + psum(bd);
                            gm = mnew;
                            if ((sb0 + 32) % grp == 0 || sb0 + 32 >= a.nslot) {
                                const float dG = gl > 0.f ? gd / gl : 0.f;
                                if (hh == 0) {
                                    sm.lsel[wave][lev][l32] = gl > 0.f ? gm + __log2f(gl) : -INFINITY;
                                    sm.ddl[wave][lev][l32] = dG;
                                    dsum += dG;
                                }
                            }
                            continue;
                        }
                        const float lg = sm.lsel[wave][lev][l32], dG = sm.ddl[wave][lev][l32];
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            const float p = lg > -INFINITY ? fexp2(s[i] - lg) : 0.f;
                            s[i] = p * (dp[i] - dG);
                        }
                        if constexpr (BF16)
                            contract_rows_tr(sm.k, kb * 32, s, lane, dqc0, dqc1);
                        else
                            contract_rows<BF16>(sm.kt, P, kb * 32, s, l32, hh, dqc0, dqc1);
                        continue;
                    }
                    if (!near) {
                        // a level's softmax and D_G inside this block; dS
                        // enters dq without the near field's normaliser
#pragma unroll
                        for (int i = 0; i < 16; ++i)
                            s[i] = sm.valid[kb * 32 + acc_row(i, hh)] != 0 ? s[i] * cs : -INFINITY;
                        float lg4[4], dg4[4];
                        const int grp = a.slot_group;
                        level_block(s, dp, grp, lg4, dg4);
                        const int sb0 = (t - m.nnear) * KT + kb * 32;   // first slot of the block
#pragma unroll
                        for (int c = 0; c < 4; ++c) {
                            // the lane that holds a group's first row records it
                            const int row0 = 8 * c + 4 * hh;
                            const bool owner = grp == 4 || (hh == 0 && (row0 & (grp - 1)) == 0);
                            const int lev = (sb0 + row0) / grp;
                            if (owner && lev < kMaxCoarse) {
                                sm.lsel[wave][lev][l32] = lg4[c];
                                sm.ddl[wave][lev][l32] = dg4[c];
                                dsum += dg4[c];
                            }
                        }
                        if constexpr (BF16)
                            contract_rows_tr(sm.k, kb * 32, s, lane, dqc0, dqc1);
                        else
                            contract_rows<BF16>(sm.kt, P, kb * 32, s, l32, hh, dqc0, dqc1);
                        continue;
                    }
                }
                const bool full = near && m.full, causal = !TWO_D && near && a.causal;
                // every row of the block visible to every query of the wave?
                const bool allvis =
                    __builtin_amdgcn_ballot_w64(!(full && (!causal || qrel >= kb * 32 + 31))) == 0;
                // masked rows' raw scores to -inf (branch-free: every row's
                // validity read, four rows per load)
                auto mask_rows = [&](f32x16 &x) {
                    if (allvis) return;
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        const int r0 = kb * 32 + 8 * c + 4 * hh;
                        const int4 v4 = *reinterpret_cast<const int4 *>(&sm.valid[r0]);
                        const int vl[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int i = 4 * c + e;
                            const bool ok = (full || vl[e] != 0) && (!causal || r0 + e <= qrel);
                            x[i] = ok ? x[i] : -INFINITY;
                        }
                    }
                };
                // P = exp2(s tau log2e - m) against the reference maximum m
                // as it stands, no block maximum (m only keeps P finite);
                // when a lane's block sum passes 2^64 (a score more than ~60
                // above m; the first block, whose m is still -1e30), the
                // block's scores are formed again, m is raised to their
                // maximum, l and dq rescaled, and P formed anew
                if constexpr (!PL) {
                    mask_rows(s);
                    float bl = 0.f;
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        s[i] = fexp2(fmaf(s[i], cs, -mrun));   // 0 for masked rows
                        bl += s[i];
                    }
                    if (__builtin_amdgcn_ballot_w64(bl > 0x1p64f) != 0) {
                        RowOp<BF16> kr2;
                        if constexpr (BF16)
                            row_from_tile(kr2, sm.k, kb * 32 + l32, hh);
                        else
                            kr2.from_lds(sm.k + (kb * 32 + l32) * P, hh);
                        f32x16 s2 = contract_channels<BF16>(kr2, qo, f32x16{0});
                        mask_rows(s2);
                        float mx = -INFINITY;
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            s2[i] *= cs;
                            mx = fmaxf(mx, s2[i]);
                        }
                        const float mnew = fmaxf(mrun, pmax(mx));
                        const float corr = fexp2(mrun - mnew);
                        lrun *= corr;
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            dq0[i] *= corr;
                            dq1[i] *= corr;
                        }
                        mrun = mnew;
                        bl = 0.f;
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            s[i] = fexp2(s2[i] - mrun);
                            bl += s[i];
                        }
                    }
                    lrun += bl;
#pragma unroll
                    for (int i = 0; i < 16; ++i) s[i] = s[i] * (dp[i] - dnear);   // dS
                } else {
                    // (per-level instances: the lazy maximum, which keeps
                    // their registers within budget)
                    mask_rows(s);
                    float mx = -INFINITY;
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        s[i] *= cs;
                        mx = fmaxf(mx, s[i]);
                    }
                    mx = pmax(mx);
                    const bool raise = mx > mrun + 8.0f;
                    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
                        const float mnew = raise ? mx : mrun;
                        const float corr = fexp2(mrun - mnew);
                        lrun *= corr;
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            dq0[i] *= corr;
                            dq1[i] *= corr;
                        }
                        mrun = mnew;
                    }
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const float p = fexp2(s[i] - mrun);   // 0 for masked rows
                        lrun += p;
                        s[i] = p * (dp[i] - dnear);
                    }
                }
                if constexpr (BF16)
                    contract_rows_tr(sm.k, kb * 32, s, lane, dq0, dq1);
                else
                    contract_rows<BF16>(sm.kt, P, kb * 32, s, l32, hh, dq0, dq1);
            }
        }
    }
    const float lsum = psum(lrun);
    const float lse = mrun + __log2f(lsum);
    {
        const float f = lsum > 0.f ? a.scale / lsum : 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            dq0[i] = dq0[i] * f + (PL ? a.scale * dqc0[i] : 0.f);
            dq1[i] = dq1[i] * f + (PL ? a.scale * dqc1[i] : 0.f);
        }
    }
    if (active && hh == 0) {
        // the key pass sees the near field's lse and D (joint: the query's);
        // a repeated query (zero dO, D = 0) keeps its own finite lse here
        if (qlive) {
            stf(a.lse, (long long)slice * a.n + qtok, a.lse_elems, lse);
            stf(a.delta, (long long)slice * a.n + qtok, a.lse_elems, dnear);
        }
        sm.lse[wave][l32] = lse;
        sm.dd[wave][l32] = dnear;
    }

    // ---- pass 2, the coarse tiles again: with the slots on the lanes (S:
    // queries x slots) the scores give this wave's part of the block's
    // dK_bar = tau Q^T dS and dV_bar = dO^T P per slot (P from the final lse).
    // The waves' parts are added in wave order through LDS (every wave takes
    // part, in workgroup-uniform control flow) and the last wave stores the
    // workgroup's partial row.
    if (tend_near < ntl) {
        KVTile<BF16, TWO_D, NT, true> kv;
        kv.fetch(a, m, b, tile_of(tend_near), slice, tid);
        for (int x = tend_near; x < ntl; ++x) {
            const int t = tile_of(x);
            __syncthreads();   // also orders sm.lse / sm.dd before their reads
            kv.stash(sm.k, sm.kt, sm.v, sm.valid, tid);
            __syncthreads();
            lin_scores(t);
            if (x + 1 < ntl) kv.fetch(a, m, b, tile_of(x + 1), slice, tid);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const int slot0 = (t - m.nnear) * KT + kb * 32;
                if (slot0 >= a.nslot) continue;   // uniform
                f32x16 s2 = {0}, p2 = {0};
                if (active) {
                    RowOp<BF16> kro, vro;
                    if constexpr (BF16) {
                        row_from_tile(kro, sm.k, kb * 32 + l32, hh);
                        row_from_tile(vro, sm.v, kb * 32 + l32, hh);
                    } else {
                        kro.from_lds(sm.k + (kb * 32 + l32) * P, hh);
                        vro.from_lds(sm.v + (kb * 32 + l32) * P, hh);
                    }
                    if constexpr (LIN)
                        s2 = f32x16{0};   // the slot's shared score is in sm.lins
                    else
                        s2 = contract_channels<BF16>(qo, kro, f32x16{0});
                    p2 = contract_channels<BF16>(go, vro, f32x16{0});   // dP, then P
                    const bool okc = sm.valid[kb * 32 + l32] != 0;
                    // branch-free: the query rows' lse and D read four at a
                    // time, empty slots zeroed by a select
                    const float *lrow = sm.lse[wave], *drow = sm.dd[wave];
                    if constexpr (PL) {
                        // this lane's slot belongs to one level: its lse and D_G
                        int lev = (slot0 + l32) / a.slot_group;
                        lev = lev < kMaxCoarse ? lev : kMaxCoarse - 1;
                        lrow = sm.lsel[wave][lev];
                        drow = sm.ddl[wave][lev];
                    }
                    const float sl = LIN ? sm.lins[kb * 32 + l32] * cs : 0.f;
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        const int r0 = 8 * c + 4 * hh;
                        const float4 l4 = *reinterpret_cast<const float4 *>(lrow + r0);
                        const float4 d4 = *reinterpret_cast<const float4 *>(drow + r0);
                        const float lv[4] = {l4.x, l4.y, l4.z, l4.w}, dv[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int i = 4 * c + e;
                            const float ex = LIN ? fexp2(sl - lv[e]) : fexp2(fmaf(s2[i], cs, -lv[e]));
                            const float pp = okc ? ex : 0.f;
                            s2[i] = pp * (p2[i] - dv[e]);   // dS
                            p2[i] = pp;
                        }
                    }
                }
                const int slot = slot0 + l32;
                const long long prow = (long long)b * gpb + gi;   // this workgroup's partial row
                // FMA-linear: c = this wave's sum of dS over its queries for the
                // lane's slot, and the slot's coarse query
                float cl = 0.f;
                int sl_set = 0;
                if constexpr (LIN) {
                    if (active) {
                        float acc = 0.f;
#pragma unroll
                        for (int i = 0; i < 16; ++i) acc += s2[i];
                        cl = psum(acc);
                    }
                    sl_set = slot / K;
                    sl_set = sl_set < kMaxCoarse ? sl_set : kMaxCoarse - 1;
                }
                const long long base0 = (((long long)ls * a.npart + prow) * a.nslot + slot) * kHeadDim;
                const long long base1 = base0 + (long long)a.pslices * a.npart * a.nslot * kHeadDim;
                if constexpr (BF16 && NW == 4 && !LIN) {
                    // four waves: every lane passes its dS column (then its P
                    // column), in bf16, through LDS; waves 0 and 1 form the
                    // two channel halves of the dK_bar partial over all four
                    // waves' queries (in wave order) on the matrix cores,
                    // waves 2 and 3 those of dV_bar, and each stores its half
                    __bf16 *const xch = reinterpret_cast<__bf16 *>(sm.cred);   // [4 waves][64 lanes][16]
#pragma unroll
                    for (int which = 0; which < 2; ++which) {
                        const f32x16 &w_ = which ? p2 : s2;
                        bf16x8 own[2];
#pragma unroll
                        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
                            for (int e = 0; e < 8; ++e) own[hf][e] = static_cast<__bf16>(w_[8 * hf + e]);
                        __syncthreads();   // the previous exchange has been read
                        *reinterpret_cast<bf16x8 *>(xch + (wave * 64 + lane) * 16) = own[0];
                        *reinterpret_cast<bf16x8 *>(xch + (wave * 64 + lane) * 16 + 8) = own[1];
                        __syncthreads();
                        if ((wave >> 1) == which) {
                            const int half = wave & 1;
                            f32x16 c = {0};
#pragma unroll
                            for (int sw = 0; sw < 4; ++sw) {
                                bf16x8 src[2];
                                src[0] = *reinterpret_cast<const bf16x8 *>(xch + (sw * 64 + lane) * 16);
                                src[1] = *reinterpret_cast<const bf16x8 *>(xch + (sw * 64 + lane) * 16 + 8);
                                c = contract_rows_tr1(which ? sm.dot[sw] : sm.qt[sw], src, lane, half, c);
                            }
                            const float f = which ? 1.0f : a.scale;
                            if (slot < a.nslot) {
#pragma unroll
                                for (int g4 = 0; g4 < 4; ++g4) {
                                    const int ch = 32 * half + 8 * g4 + 4 * hh;
                                    st4f(a.part, (which ? base1 : base0) + ch, a.part_elems, f * c[4 * g4],
                                         f * c[4 * g4 + 1], f * c[4 * g4 + 2], f * c[4 * g4 + 3]);
                                }
                            }
                        }
                    }
                } else if constexpr (BF16 && NW == 2 && !LIN) {
                    // two waves: each lane passes its dS (then P) column, in
                    // bf16, to the same lane of the other wave through LDS, and
                    // wave w forms channel half w of the partial over both
                    // waves' queries (its own first) on the matrix cores,
                    // then stores it: no wave-by-wave sums
                    __bf16 *const xch = reinterpret_cast<__bf16 *>(sm.cred);   // [2 waves][64 lanes][16]
#pragma unroll
                    for (int which = 0; which < 2; ++which) {
                        const f32x16 &w_ = which ? p2 : s2;
                        bf16x8 own[2], oth[2];
#pragma unroll
                        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
                            for (int e = 0; e < 8; ++e) own[hf][e] = static_cast<__bf16>(w_[8 * hf + e]);
                        __syncthreads();   // the other wave has read the previous exchange
                        *reinterpret_cast<bf16x8 *>(xch + (wave * 64 + lane) * 16) = own[0];
                        *reinterpret_cast<bf16x8 *>(xch + (wave * 64 + lane) * 16 + 8) = own[1];
                        __syncthreads();
                        oth[0] = *reinterpret_cast<const bf16x8 *>(xch + ((wave ^ 1) * 64 + lane) * 16);
                        oth[1] = *reinterpret_cast<const bf16x8 *>(xch + ((wave ^ 1) * 64 + lane) * 16 + 8);
                        f32x16 c = {0};
                        c = contract_rows_tr1(which ? sm.dot[wave] : sm.qt[wave], own, lane, wave, c);
                        c = contract_rows_tr1(which ? sm.dot[wave ^ 1] : sm.qt[wave ^ 1], oth, lane, wave, c);
                        const float f = which ? 1.0f : a.scale;
                        if (slot < a.nslot) {
#pragma unroll
                            for (int g4 = 0; g4 < 4; ++g4) {
                                const int ch = 32 * wave + 8 * g4 + 4 * hh;
                                st4f(a.part, (which ? base1 : base0) + ch, a.part_elems, f * c[4 * g4],
                                     f * c[4 * g4 + 1], f * c[4 * g4 + 2], f * c[4 * g4 + 3]);
                            }
                        }
                    }
                } else {
                // one partial at a time: Q^T dS (dK_bar), then dO^T P (dV_bar);
                // the waves' parts are added half a row (32 channels) at a time
#pragma unroll
                for (int which = 0; which < 2; ++which) {
                    f32x16 c0 = {0}, c1 = {0};
                    if (LIN && which == 0) {
                        // dK_bar part: c times the slot's coarse query
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            const int ch = acc_row(i, hh);
                            c0[i] = cl * sm.qbl[sl_set][ch];
                            c1[i] = cl * sm.qbl[sl_set][32 + ch];
                        }
                    } else if (active) {
                        if constexpr (BF16)
                            contract_rows_tr(which ? sm.dot[wave] : sm.qt[wave], 0, which ? p2 : s2, lane, c0, c1);
                        else
                            contract_rows<BF16>(which ? sm.dot[wave] : sm.qt[wave], PQ, 0, which ? p2 : s2, l32, hh,
                                                c0, c1);
                    }
                    const float f = which ? 1.0f : a.scale;
                    const long long bs = which ? base1 : base0;
                    constexpr int NH = NW >= 4 ? 1 : 2;         // rounds: a whole row, or two half rows
                    constexpr int PCR = NW >= 4 ? 68 : 36;      // LDS pitch (fp32) of a slot row
                    float *const cr = sm.cred + l32 * PCR + 4 * hh;   // this lane's slot row
#pragma unroll
                    for (int hr = 0; hr < NH; ++hr) {
#pragma unroll 1
                        for (int w = 0; w < NW; ++w) {
                            if (wave == w) {
#pragma unroll
                                for (int hx = 0; hx < 2 / NH; ++hx) {
                                    const int half = NH == 2 ? hr : hx;   // channels 32 half .. 32 half + 31
                                    f32x16 &c = half ? c1 : c0;
                                    float *const crh = cr + (NH == 2 ? 0 : 32 * half);
                                    if (w > 0) {
#pragma unroll
                                        for (int g4 = 0; g4 < 4; ++g4) {
                                            const f32x4 u = *reinterpret_cast<const f32x4 *>(crh + 8 * g4);
#pragma unroll
                                            for (int e2 = 0; e2 < 4; ++e2) c[4 * g4 + e2] = u[e2] + c[4 * g4 + e2];
                                        }
                                    }
                                    if (w + 1 < NW) {
#pragma unroll
                                        for (int g4 = 0; g4 < 4; ++g4)
                                            *reinterpret_cast<f32x4 *>(crh + 8 * g4) =
                                                f32x4{c[4 * g4], c[4 * g4 + 1], c[4 * g4 + 2], c[4 * g4 + 3]};
                                    } else if (slot < a.nslot) {
#pragma unroll
                                        for (int g4 = 0; g4 < 4; ++g4) {
                                            const int ch = 32 * half + 8 * g4 + 4 * hh;
                                            st4f(a.part, bs + ch, a.part_elems, f * c[4 * g4], f * c[4 * g4 + 1],
                                                 f * c[4 * g4 + 2], f * c[4 * g4 + 3]);
                                        }
                                    }
                                }
                            }
                            __syncthreads();
                        }
                    }
                }
                }
                if constexpr (LIN) {
                    // dQ_bar of each set += c_g k_bar_g over the block's slots,
                    // c_g summed over the waves in wave order (lane = channel)
                    if (hh == 0) sm.cw[wave][l32] = cl;
                    __syncthreads();
                    if (tid < kHeadDim) {
                        for (int j = 0; j < 32 && slot0 + j < a.nslot; ++j) {
                            float c = 0.f;
                            for (int w = 0; w < NW; ++w) c += sm.cw[w][j];
                            int e = (slot0 + j) / K;
                            e = e < kMaxCoarse ? e : kMaxCoarse - 1;
                            const int row = kb * 32 + j;
                            float kv;
                            if constexpr (BF16)
                                kv = static_cast<float>(sm.k[sw_off(row, tid >> 3) + (tid & 7)]);
                            else
                                kv = sm.k[row * P + tid];
                            sm.dqb[e][tid] += c * kv;
                        }
                    }
                    __syncthreads();
                }
            }
        }
    }
    if constexpr (LIN) {
        // this workgroup's dQ_bar partial row of every set
        __syncthreads();
        const long long prow = (long long)b * gpb + gi;
        for (int x = tid; x < a.lv.nlev * kHeadDim; x += NT) {
            const int e = x / kHeadDim, ch = x - (x / kHeadDim) * kHeadDim;
            stf(a.qpart, (((long long)slice * a.npart + prow) * a.lv.nlev + e) * kHeadDim + ch, a.qpart_elems,
                a.scale * sm.dqb[e][ch]);
        }
    }
    if (!qlive) return;
    // dQ^T: channel rows, this lane's query column (tau / l already applied);
    // FMA-linear: the near field's part, in fp32, for bwd_qapply
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
        const int ch = 8 * g4 + 4 * hh;
        if constexpr (LIN) {
            st4f(a.dqn, qrow + ch, a.dqn_elems, dq0[4 * g4], dq0[4 * g4 + 1], dq0[4 * g4 + 2], dq0[4 * g4 + 3]);
            st4f(a.dqn, qrow + 32 + ch, a.dqn_elems, dq1[4 * g4], dq1[4 * g4 + 1], dq1[4 * g4 + 2],
                 dq1[4 * g4 + 3]);
        } else {
            st4<BF16>(a.dq, qrow + ch, a.io_elems, dq0[4 * g4], dq0[4 * g4 + 1], dq0[4 * g4 + 2], dq0[4 * g4 + 3]);
            st4<BF16>(a.dq, qrow + 32 + ch, a.io_elems, dq1[4 * g4], dq1[4 * g4 + 1], dq1[4 * g4 + 2],
                      dq1[4 * g4 + 3]);
        }
    }
}

// Sums of partial rows, one wave per output row: the terms, numbered in a
// fixed order, are dealt round-robin to NG groups of 64 / NG lanes (a lane
// takes eight channels), so NG partial rows are in flight per load.
// deal_box calls f(dx, dy, k) for the terms of an nx x ny x nk box (k
// fastest) numbered t0, t0 + 1, ... that fall to group grp, in ascending
// order; the caller advances t0 by the box's size.
template <int NG, typename F>
__device__ inline void deal_box(int nx, int ny, int nk, int grp, int t0, F f)
{
    const int nt = nx * ny * nk;
    int w = (grp - t0) & (NG - 1);   // this group's first term of the box
    int k = w % nk, dy = (w / nk) % ny, dx = (w / nk) / ny;
    for (; w < nt; w += NG) {
        f(dx, dy, k);
        k += NG;   // NG terms on
        while (k >= nk) {
            k -= nk;
            ++dy;
        }
        while (dy >= ny) {
            dy -= ny;
            ++dx;
        }
    }
}

// acc[i] += the eight floats at p (16-byte aligned), bounds-checked
__device__ inline void add8(float acc[8], const float *p, long long idx, long long lim)
{
    const uint4 p0 = ld16(p, idx, 4, lim), p1 = ld16(p, idx + 4, 4, lim);
    acc[0] += __uint_as_float(p0.x);
    acc[1] += __uint_as_float(p0.y);
    acc[2] += __uint_as_float(p0.z);
    acc[3] += __uint_as_float(p0.w);
    acc[4] += __uint_as_float(p1.x);
    acc[5] += __uint_as_float(p1.y);
    acc[6] += __uint_as_float(p1.z);
    acc[7] += __uint_as_float(p1.w);
}

// The eight groups' sums (lanes 8 grp + x hold channels 8 x ..): lanes of
// group 0 end with ((g0 + g1) + (g2 + g3)) + ((g4 + g5) + (g6 + g7)) and
// store them.
__device__ inline void store_group_sums(float acc[8], int grp, float *dst, long long o, long long lim)
{
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        float x = acc[i];
        x += __shfl_xor(x, 8);
        x += __shfl_xor(x, 16);
        x += __shfl_xor(x, 32);
        acc[i] = x;
    }
    if (grp == 0) {
        st4f(dst, o, lim, acc[0], acc[1], acc[2], acc[3]);
        st4f(dst, o + 4, lim, acc[4], acc[5], acc[6], acc[7]);
    }
}

// One workgroup (one wave) per (tensor, slice, coarse row).  The query
// groups whose interaction list holds the row lie within 3 groups of it
// along each axis (the list is the parent's 6-wide window); the first
// threads find, for each candidate, the list entry j that names the row (or
// none).  The partials of the chunks of those query groups, in the order
// (candidate, block, chunk), are dealt out round-robin to eight groups of
// eight lanes (lane = eight channels, two 16-byte loads per partial), so
// that eight partial rows are in flight per load; each group adds its terms
// in that order and the groups' sums are added by three exchanges and
// stored by group 0.  Slot of entry j of set e: slot_of.
// FMA-linear, dQ_bar: one wave per (slice, coarse row of set e, group g):
// the partial rows of the query-pass workgroups of the blocks (2D: cells)
// inside group g, in ascending (block, workgroup) order, dealt to eight
// lane groups as in bwd_reduce.
template <bool TWO_D>
__global__ __launch_bounds__(64) void bwd_qreduce(BwdArgs a)
{
    const long long wg = blockIdx.x;
    const int tid = threadIdx.x;
    const int slice = (int)(wg / a.R);
    const int crow = (int)(wg - (long long)slice * a.R);
    if (slice >= a.nslice) return;
    int e = 0;
    while (e + 1 < a.lv.nlev && a.lv.off[e + 1] <= crow) ++e;
    const int My = a.lv.My[e], span = 1 << (a.lv.lvl[e] - 1);
    const int g = crow - a.lv.off[e];
    const int gpb = a.npart / a.nblocks;
    const int grp = tid >> 3, c8 = (tid & 7) * 8;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int cx0, cy0, nx, ny;
    if constexpr (TWO_D) {
        cx0 = (g / My) * span;
        cy0 = (g - (g / My) * My) * span;
        nx = a.nbx - cx0 < span ? a.nbx - cx0 : span;
        ny = a.nby - cy0 < span ? a.nby - cy0 : span;
    } else {
        cx0 = g * span;
        cy0 = 0;
        nx = a.nblocks - cx0 < span ? a.nblocks - cx0 : span;
        ny = 1;
    }
    deal_box<8>(nx, ny, gpb, grp, 0, [&](int dx, int dy, int k) {
        const long long prow = TWO_D ? (long long)((cx0 + dx) * a.nby + cy0 + dy) * gpb + k
                                     : (long long)(cx0 + dx) * gpb + k;
        add8(acc, a.qpart, (((long long)slice * a.npart + prow) * a.lv.nlev + e) * kHeadDim + c8, a.qpart_elems);
    });
    store_group_sums(acc, grp, a.dqbar, ((long long)slice * a.R + crow) * kHeadDim + c8, a.coarse_elems);
}

// FMA-linear, dq: eight lanes per token, eight channels per lane, 32 tokens
// per workgroup (workgroup = (slice, run of 32 tokens)): the near field's
// part plus pi^q * dQ_bar of the token's group of every set, stored in the
// I/O dtype; and q_t . dQ_bar per set for dpi^q (each lane's eight products,
// then the eight lanes of the token added with three exchanges).  The
// launcher keeps tokens per slice and the workgroup count below 2^31.
template <bool BF16, bool TWO_D>
__global__ __launch_bounds__(256) void bwd_qapply(BwdArgs a, int runs)
{
    const int slice = (int)(blockIdx.x / (unsigned)runs);
    const int t = ((int)blockIdx.x - slice * runs) * 32 + (int)(threadIdx.x >> 3);
    const int c8 = (int)(threadIdx.x & 7) * 8;
    const bool live = slice < a.nslice && t < a.n;
    const long long row = ((long long)slice * a.n + t) * kHeadDim + c8;
    const long long lim = live ? a.io_elems : 0;
    float acc[8], qv[8];
    {
        const uint4 n0 = ld16(a.dqn, row, 4, live ? a.dqn_elems : 0);
        const uint4 n1 = ld16(a.dqn, row + 4, 4, live ? a.dqn_elems : 0);
        acc[0] = __uint_as_float(n0.x); acc[1] = __uint_as_float(n0.y);
        acc[2] = __uint_as_float(n0.z); acc[3] = __uint_as_float(n0.w);
        acc[4] = __uint_as_float(n1.x); acc[5] = __uint_as_float(n1.y);
        acc[6] = __uint_as_float(n1.z); acc[7] = __uint_as_float(n1.w);
    }
    if constexpr (BF16) {
        const uint4 w = ld16(a.q, row, 2, lim);
        const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            qv[2 * i] = bf16lo_to_f32(u[i]);
            qv[2 * i + 1] = bf16hi_to_f32(u[i]);
        }
    } else {
        const uint4 w0 = ld16(a.q, row, 4, lim), w1 = ld16(a.q, row + 4, 4, lim);
        qv[0] = __uint_as_float(w0.x); qv[1] = __uint_as_float(w0.y);
        qv[2] = __uint_as_float(w0.z); qv[3] = __uint_as_float(w0.w);
        qv[4] = __uint_as_float(w1.x); qv[5] = __uint_as_float(w1.y);
        qv[6] = __uint_as_float(w1.z); qv[7] = __uint_as_float(w1.w);
    }
    const int hw = a.w_stride ? slice % a.heads : 0;
    const long long wbase = (long long)hw * a.wlen;
    int x = 0, y = 0;
    if constexpr (TWO_D) {
        x = t / a.side;
        y = t - x * a.side;
    }
    for (int e = 0; e < a.lv.nlev; ++e) {
        const int s = a.lv.size[e];
        int g;
        float w;
        if constexpr (TWO_D) {
            const int gx = x / s, gy = y / s;
            g = gx * a.lv.My[e] + gy;
            w = ldf(a.wq, live ? wbase + a.lv.woff[e] + (x - gx * s) : -1, a.w_elems) *
                ldf(a.wq, live ? wbase + a.lv.woff[e] + s + (y - gy * s) : -1, a.w_elems);
        } else {
            g = t / s;
            w = ldf(a.wq, live ? wbase + a.lv.woff[e] + (t - g * s) : -1, a.w_elems);
        }
        const long long drow = ((long long)slice * a.R + a.lv.off[e] + g) * kHeadDim + c8;
        const long long dlim = live ? a.coarse_elems : 0;
        const uint4 d0 = ld16(a.dqbar, drow, 4, dlim), d1 = ld16(a.dqbar, drow + 4, 4, dlim);
        const float d[8] = {__uint_as_float(d0.x), __uint_as_float(d0.y), __uint_as_float(d0.z),
                            __uint_as_float(d0.w), __uint_as_float(d1.x), __uint_as_float(d1.y),
                            __uint_as_float(d1.z), __uint_as_float(d1.w)};
        float dot = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            acc[i] += w * d[i];
            dot += qv[i] * d[i];
        }
        dot += __shfl_xor(dot, 1);
        dot += __shfl_xor(dot, 2);
        dot += __shfl_xor(dot, 4);
        if ((threadIdx.x & 7) == 0 && live)
            stf(a.dotq, ((long long)slice * a.lv.nlev + e) * a.n + t, a.dot_elems, dot);
    }
    st4<BF16>(a.dq, row, lim, acc[0], acc[1], acc[2], acc[3]);
    st4<BF16>(a.dq, row + 4, lim, acc[4], acc[5], acc[6], acc[7]);
}

// Slot of entry j of coarse set e in a block's list (inverse of coarse_source).
template <bool TWO_D>
__device__ inline int slot_of(const BwdArgs &a, int e, int j)
{
    constexpr int K = TWO_D ? kSlots2D : kSlots1D;
    if (a.norm_level) return (e / a.rank) * a.slot_group + (e - (e / a.rank) * a.rank) * K + j;
    return e * K + j;
}

// --------------------------------------------------------------- bwd_reduce
// The entry j of level group (qx, qy)'s 2D list that names square (u, v)
// of the same level, or -1: the inverse of list2d_entry (the square's place
// in the row-major 6x6 window around the parent, skipping the 3x3 block at
// (1 + (qx & 1), 1 + (qy & 1)); see window_slot), for squares inside the map.
__device__ inline int list2d_slot_of(int qx, int qy, int u, int v)
{
    const int au = u - (2 * (qx >> 1) - 2), av = v - (2 * (qy >> 1) - 2);
    if (au < 0 || au >= 6 || av < 0 || av >= 6) return -1;
    const int ox = 1 + (qx & 1), oy = 1 + (qy & 1);
    if (au < ox) return au * 6 + av;
    if (au < ox + 3) {
        if (av >= oy && av < oy + 3) return -1;   // the finer levels' squares
        return 6 * ox + (au - ox) * 3 + (av < oy ? av : av - 3);
    }
    return 6 * ox + 9 + (au - ox - 3) * 6 + av;
}

template <bool TWO_D>
__global__ __launch_bounds__(64) void bwd_reduce(BwdArgs a)
{
    constexpr int K = TWO_D ? kSlots2D : kSlots1D;
    constexpr int NC = TWO_D ? 49 : 7;       // candidate query groups: 7 per axis
    __shared__ int cand_j[NC];
    const long long wg = blockIdx.x;
    const int tid = threadIdx.x;
    const int z = (int)(wg / ((long long)a.pslices * a.R));
    const long long rem = wg - (long long)z * a.pslices * a.R;
    const int ls = (int)(rem / a.R);   // slice within the pass
    const int crow = (int)(rem - (long long)ls * a.R);
    const int slice = a.slice0 + ls;
    if (z > 1 || slice >= a.nslice) return;
    int e = 0;
    while (e + 1 < a.lv.nlev && a.lv.off[e + 1] <= crow) ++e;
    const int lvl = a.lv.lvl[e], M = a.lv.M[e], My = a.lv.My[e];
    const int g = crow - a.lv.off[e];
    const int span = 1 << (lvl - 1);          // base blocks (cells per side) per level group
    const int gpb = a.npart / a.nblocks;      // partial rows per query block
    const int u = TWO_D ? g / My : g, v = TWO_D ? g - (g / My) * My : 0;
    if (tid < NC) {
        int jj = -1;
        if constexpr (TWO_D) {
            const int qx = u - 3 + tid / 7, qy = v - 3 + tid % 7;
            if (qx >= 0 && qy >= 0 && qx < M && qy < My && qx * span < a.nbx && qy * span < a.nby)
                jj = list2d_slot_of(qx, qy, u, v);
        } else {
            const int q = g - 3 + tid;
            if (q >= 0 && q < M && q * span < a.nblocks)
                for (int j = 0; j < K; ++j)
                    if (list1d_entry(q * span, lvl, j, M, a.causal) == g) jj = j;
        }
        cand_j[tid] = jj;
    }
    __syncthreads();
    const int grp = tid >> 3, c8 = (tid & 7) * 8;
    const long long zoff = (long long)z * a.pslices * a.npart * a.nslot * kHeadDim;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int t0 = 0;   // running index of the candidate's first term
    for (int c = 0; c < NC; ++c) {
        const int j = cand_j[c];
        if (j < 0) continue;
        const int slot = slot_of<TWO_D>(a, e, j);
        int cx0, cy0, nx, ny;
        if constexpr (TWO_D) {
            cx0 = (u - 3 + c / 7) * span;
            cy0 = (v - 3 + c % 7) * span;
            nx = a.nbx - cx0 < span ? a.nbx - cx0 : span;
            ny = a.nby - cy0 < span ? a.nby - cy0 : span;
        } else {
            cx0 = (g - 3 + c) * span;
            cy0 = 0;
            nx = a.nblocks - cx0 < span ? a.nblocks - cx0 : span;
            ny = 1;
        }
        // terms: (cell row dx, cell column dy, chunk k)
        deal_box<8>(nx, ny, gpb, grp, t0, [&](int dx, int dy, int k) {
            const long long ck = TWO_D ? (long long)((cx0 + dx) * a.nby + cy0 + dy) * gpb + k
                                       : (long long)(cx0 + dx) * gpb + k;
            add8(acc, a.part, zoff + (((long long)ls * a.npart + ck) * a.nslot + slot) * kHeadDim + c8, a.part_elems);
        });
        t0 += nx * ny * gpb;
    }
    store_group_sums(acc, grp, z ? a.dvbar : a.dkbar, ((long long)slice * a.R + crow) * kHeadDim + c8,
                     a.coarse_elems);
}

// --------------------------------------------------------------- bwd_key
template <bool BF16>
struct KSmem {
    typedef typename Elt<BF16>::T T;
    T q[KT * Elt<BF16>::P];
    T qt[BF16 ? 8 : kHeadDim * Elt<BF16>::P];   // fp32 only: Q transposed
    T g[KT * Elt<BF16>::P];
    T gt[BF16 ? 8 : kHeadDim * Elt<BF16>::P];   // fp32 only: dO transposed
    // per query row; lse = +inf for rows past the map / sequence (read four
    // rows at a time)
    __attribute__((aligned(16))) float lse[KT];
    __attribute__((aligned(16))) float dd[KT];
    float cbar[2][kHeadDim];   // dK_bar, dV_bar row of one coarse set
};

// A key block's near window of queries: 1D the tokens [qlo, qhi); 2D the
// in-map 3x3 cells (tpc tiles each, or packed 64 tokens to a tile when a
// cell is smaller than a tile: full = false).
struct QWin {
    long long qlo, qhi;
    Near2D nd;
    int tpc, csz, lg;
    bool full;
};

// One 64-query tile of a key block's near window in registers: Q and dO
// rows (NT threads, 16 bytes each per load) plus lse, D and the token of
// every row; stash() writes them to LDS (bf16: swizzled rows; fp32: rows
// and transposes).
template <bool BF16, bool TWO_D, int NT>
struct QTile {
    typedef typename Elt<BF16>::T T;
    static constexpr int PER = Elt<BF16>::PER16, CPR = kHeadDim / PER, P = Elt<BF16>::P;
    static constexpr int ITER = KT * CPR / NT;
    static_assert(KT * CPR % NT == 0 && NT >= KT, "tile split");
    uint4 qr[ITER], gr[ITER];
    long long tok;         // row tid's token (tid < 64)
    float lse, dd;

    // token of row `row` of tile t, or -1 past the window: 1D qlo + 64 t +
    // row below qhi; 2D pixel pofs + row of the tile's cell, whose first token
    // (base) and pofs are the tile's uniform part, formed once per tile (cells
    // smaller than a tile: position 64 t + row of the cells' tokens, cell
    // after cell)
    __device__ void tile_base(const BwdArgs &a, int t, const QWin &q, long long &base, int &pofs) const
    {
        base = 0;
        pofs = 0;
        if constexpr (TWO_D) {
            if (q.full) {
                const int ci = t / q.tpc;
                pofs = (t - ci * q.tpc) * KT;
                base = near2d_token(a, q.nd, ci, 0, q.lg);
            }
        } else {
            base = q.qlo + (long long)t * KT;
        }
    }
    __device__ long long row_token(const BwdArgs &a, const QWin &q, int t, long long base, int pofs, int row) const
    {
        if constexpr (TWO_D) {
            if (q.full) {
                const int p = pofs + row;
                return base + (long long)(p >> q.lg) * a.side + (p & (a.r - 1));
            }
            const int pg = t * KT + row, ci = pg / q.csz;
            return ci < q.nd.ncell ? near2d_token(a, q.nd, ci, pg - ci * q.csz, q.lg) : -1;
        } else {
            return base + row < q.qhi ? base + row : -1;
        }
    }

    __device__ void fetch(const BwdArgs &a, int t, int slice, const QWin &q, int tid)
    {
        constexpr int ES = BF16 ? 2 : 4;
        long long base;
        int pofs;
        tile_base(a, t, q, base, pofs);
#pragma unroll
        for (int it = 0; it < ITER; ++it) {
            const int c = tid + it * NT;
            const int row = c / CPR, col = c - (c / CPR) * CPR;
            const long long rt = row_token(a, q, t, base, pofs, row);
            const long long e = rt >= 0 ? ((long long)slice * a.n + rt) * kHeadDim + col * PER : -1;
            qr[it] = ld16(a.q, e, ES, a.io_elems);
            gr[it] = ld16(a.dout, e, ES, a.io_elems);
        }
        if (tid < KT) {
            tok = row_token(a, q, t, base, pofs, tid);
            lse = tok >= 0 ? ldf(a.lse, (long long)slice * a.n + tok, a.lse_elems) : 0.f;
            dd = tok >= 0 ? ldf(a.delta, (long long)slice * a.n + tok, a.lse_elems) : 0.f;
        }
    }

    __device__ void stash(KSmem<BF16> &sm, const BwdArgs &a, int tid) const
    {
#pragma unroll
        for (int it = 0; it < ITER; ++it) {
            const int c = tid + it * NT;
            const int row = c / CPR, col = c - (c / CPR) * CPR;
            const int o = BF16 ? sw_off(row, col) : row * P + col * PER;
            *reinterpret_cast<uint4 *>(sm.q + o) = qr[it];
            *reinterpret_cast<uint4 *>(sm.g + o) = gr[it];
            if constexpr (!BF16) {
                const T *qv = reinterpret_cast<const T *>(&qr[it]);
                const T *gv = reinterpret_cast<const T *>(&gr[it]);
#pragma unroll
                for (int e = 0; e < PER; ++e) {
                    sm.qt[(col * PER + e) * P + row] = qv[e];
                    sm.gt[(col * PER + e) * P + row] = gv[e];
                }
            }
        }
        if (tid < KT) {
            sm.lse[tid] = tok >= 0 && tok < a.n ? lse : INFINITY;
            sm.dd[tid] = dd;
        }
    }
};

// One workgroup = NW waves of one key block, wave w taking the block's
// 32-key chunk g * NW + w (waves past the block's chunks only help to load);
// the query tiles of the block's near window are loaded once for all waves,
// the next one into registers while the current one is multiplied out.
// bf16: registers for two waves per SIMD, as bwd_query
template <bool BF16, bool TWO_D, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(BF16 && (TWO_D || NW >= 4) ? 2 : 1))) void bwd_key(BwdArgs a)
{
    constexpr int NT = 64 * NW;
    constexpr int ES = BF16 ? 2 : 4;
    constexpr int P = Elt<BF16>::P;
    __shared__ __attribute__((aligned(16))) KSmem<BF16> sm;
    const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hh = lane >> 5;
    const int wave = tid >> 6;
    const int cpb = (a.qtile + 31) / 32;
    const int gpb = (cpb + NW - 1) / NW;
    const long long wg = blockIdx.x;
    const int slice = (int)(wg / ((long long)a.nblocks * gpb));
    const long long rem = wg - (long long)slice * a.nblocks * gpb;
    const int b = (int)(rem / gpb), gi = (int)(rem - (rem / gpb) * gpb);
    if (slice >= a.nslice) return;
    const int cw = gi * NW + wave;
    const bool active = cw < cpb;
    // lanes past a block smaller than the wave repeat one of its keys and
    // store nothing
    const bool klive = active && cw * 32 + l32 < a.qtile;

    // this lane's key and its K, V operands (B side)
    const long long ktok = active ? block_tok<TWO_D>(a, b, klive ? cw * 32 + l32 : l32 % a.qtile) : 0;
    const long long krow = ((long long)slice * a.n + ktok) * kHeadDim;
    RowOp<BF16> ko, vo;
    if constexpr (BF16) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            ko.x[c] = __builtin_bit_cast(bf16x8, ld16(a.k, krow + 16 * c + 8 * hh, ES, a.io_elems));
            vo.x[c] = __builtin_bit_cast(bf16x8, ld16(a.v, krow + 16 * c + 8 * hh, ES, a.io_elems));
        }
    } else {
#pragma unroll
        for (int c = 0; c < 32; ++c) {
            ko.x[c] = ldf(static_cast<const float *>(a.k), krow + 2 * c + hh, a.io_elems);
            vo.x[c] = ldf(static_cast<const float *>(a.v), krow + 2 * c + hh, a.io_elems);
        }
    }
    const float cs = a.scale_log2;

    // query tiles of the near window: 1D the token range [qlo, qhi), 2D the
    // in-map 3x3 cells, qtile / 64 tiles each (or packed)
    QWin qw;
    qw.qlo = qw.qhi = 0;
    qw.nd = Near2D{0, 0, 1, 0};
    qw.csz = a.qtile;
    qw.tpc = a.qtile / KT;
    qw.lg = 31 - __builtin_clz(a.r);
    int ntile;
    if constexpr (TWO_D) {
        qw.nd = near2d(a, b);
        qw.full = qw.csz % KT == 0;
        ntile = (qw.nd.ncell * qw.csz + KT - 1) / KT;
    } else {
        // causal: queries at or after the workgroup's first key
        qw.qlo = a.causal ? (long long)b * a.r + (long long)gi * NW * 32 / KT * KT
                          : (b > 0 ? (long long)(b - 1) * a.r : 0);
        qw.qhi = (long long)(b + 2) * a.r;
        if (qw.qhi > a.n) qw.qhi = a.n;
        qw.full = true;
        ntile = qw.qhi > qw.qlo ? (int)((qw.qhi - qw.qlo + KT - 1) / KT) : 0;
    }
    const long long qlo = qw.qlo;

    f32x16 dk0 = {0}, dk1 = {0}, dv0 = {0}, dv1 = {0};
    {
        QTile<BF16, TWO_D, NT> qt;
        if (ntile > 0) qt.fetch(a, 0, slice, qw, tid);
        for (int t = 0; t < ntile; ++t) {
            __syncthreads();
            qt.stash(sm, a, tid);
            __syncthreads();
            if (t + 1 < ntile) qt.fetch(a, t + 1, slice, qw, tid);
            if (!active) continue;
            // 1D causal: tile row r (token qlo + 64 t + r) sees this key iff r >= rmin
            const long long kd = ktok - (qlo + (long long)t * KT);
            const int rmin = (TWO_D || !a.causal) ? 0 : kd < 0 ? 0 : kd > KT ? KT : (int)kd;
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                RowOp<BF16> qro, gro;
                if constexpr (BF16) {
                    row_from_tile(qro, sm.q, qb * 32 + l32, hh);
                    row_from_tile(gro, sm.g, qb * 32 + l32, hh);
                } else {
                    qro.from_lds(sm.q + (qb * 32 + l32) * P, hh);
                    gro.from_lds(sm.g + (qb * 32 + l32) * P, hh);
                }
                f32x16 s = contract_channels<BF16>(qro, ko, f32x16{0});    // S: queries x keys
                f32x16 dp = contract_channels<BF16>(gro, vo, f32x16{0});   // dP
                f32x16 p;
                // branch-free: every row's lse and D read (four rows per
                // load), the causal rows before rmin zeroed by a select
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int r0 = qb * 32 + 8 * c + 4 * hh;
                    const float4 l4 = *reinterpret_cast<const float4 *>(&sm.lse[r0]);
                    const float4 d4 = *reinterpret_cast<const float4 *>(&sm.dd[r0]);
                    const float lv[4] = {l4.x, l4.y, l4.z, l4.w}, dv[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int i = 4 * c + e;
                        const float ex = fexp2(fmaf(s[i], cs, -lv[e]));   // 0 for rows with lse = +inf
                        p[i] = TWO_D || r0 + e >= rmin ? ex : 0.f;
                        s[i] = p[i] * (dp[i] - dv[e]);                     // dS
                    }
                }
                if constexpr (BF16) {
                    contract_rows_tr(sm.g, qb * 32, p, lane, dv0, dv1);   // dO^T P
                    contract_rows_tr(sm.q, qb * 32, s, lane, dk0, dk1);   // Q^T dS
                } else {
                    contract_rows<BF16>(sm.gt, P, qb * 32, p, l32, hh, dv0, dv1);
                    contract_rows<BF16>(sm.qt, P, qb * 32, s, l32, hh, dk0, dk1);
                }
            }
        }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        dk0[i] *= a.scale;
        dk1[i] *= a.scale;
    }

    // coarse sets: dk += pi^k * dK_bar, dv += pi^v * dV_bar of the key's group,
    // and the dot products for the weight gradients.  Every key of the block
    // lies in the same group of every set.
    const int hw = a.w_stride ? slice % a.heads : 0;
    const long long wbase = (long long)hw * a.wlen;
    const long long btok = block_tok<TWO_D>(a, b, 0);
    if constexpr (BF16) {
        // On the matrix cores, 16 sets at a time (k slots = sets):
        //   dk^T += dK_bar^T W^k and dv^T += dV_bar^T W^v (rows channels,
        //   columns keys), with dK_bar, dV_bar and the weights split into a
        //   bf16 high part and the bf16 rounding of the rest, summed as
        //   hi*hi + lo*hi + hi*lo (error ~2^-17 of each product);
        //   dot_k[e][key] = dK_bar_e . k (rows sets, columns keys, k slots the
        //   channels; k is exact in bf16, dK_bar enters as hi + lo).
        // The query tiles' LDS holds the operands: ca = [tensor][hi, lo][64
        // channels][16 sets], cb = [tensor][hi, lo][16 sets][PB].
        __bf16 *const ca = sm.q;
        __bf16 *const cb = sm.g;
        // s_l = r 2^(l-1): the block's level-l group is b >> (l-1) (2D: per
        // axis, cell >> (l-1)), and the key's offset in it (b mod 2^(l-1)) r
        // plus its position in the block (2D: per axis)
        const int kp = klive ? cw * 32 + l32 : l32 % a.qtile;
        int bcx = b, bcy = 0, kpx = kp, kpy = 0;
        if constexpr (TWO_D) {
            bcx = b / a.nby;
            bcy = b - bcx * a.nby;
            kpx = kp / a.r;
            kpy = kp - kpx * a.r;
        }
        for (int e0 = 0; e0 < a.lv.nlev; e0 += 16) {
            __syncthreads();   // the tiles, or the previous chunk's operands, are no longer read
            for (int it = tid; it < 256; it += NT) {
                const int z = it >> 7, el = (it >> 3) & 15, c8 = (it & 7) * 8;
                const int e = e0 + el;
                float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
                if (e < a.lv.nlev) {
                    const int sh = a.lv.lvl[e] - 1;
                    const int gb = TWO_D ? (bcx >> sh) * a.lv.My[e] + (bcy >> sh) : bcx >> sh;
                    const long long rb = ((long long)slice * a.R + a.lv.off[e] + gb) * kHeadDim + c8;
                    const float *src = z ? a.dvbar : a.dkbar;
                    const uint4 u0 = ld16(src, rb, 4, a.coarse_elems), u1 = ld16(src, rb + 4, 4, a.coarse_elems);
                    x[0] = __uint_as_float(u0.x); x[1] = __uint_as_float(u0.y);
                    x[2] = __uint_as_float(u0.z); x[3] = __uint_as_float(u0.w);
                    x[4] = __uint_as_float(u1.x); x[5] = __uint_as_float(u1.y);
                    x[6] = __uint_as_float(u1.z); x[7] = __uint_as_float(u1.w);
                }
                bf16x8 h, l;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    h[j] = static_cast<__bf16>(x[j]);
                    l[j] = static_cast<__bf16>(x[j] - static_cast<float>(h[j]));
                }
                *reinterpret_cast<bf16x8 *>(cb + ((z * 2 + 0) * 16 + el) * PB + c8) = h;
                *reinterpret_cast<bf16x8 *>(cb + ((z * 2 + 1) * 16 + el) * PB + c8) = l;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    ca[((z * 2 + 0) * kHeadDim + c8 + j) * 16 + el] = h[j];
                    ca[((z * 2 + 1) * kHeadDim + c8 + j) * 16 + el] = l[j];
                }
            }
            __syncthreads();
            if (!active) continue;
            // this lane's key: the weights of sets e0 + 8 hh .. + 7 (B operand)
            bf16x8 wkh, wkl, wvh, wvl;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int e = e0 + 8 * hh + j;
                float wk = 0.f, wv = 0.f;
                if (e < a.lv.nlev) {
                    const int sh = a.lv.lvl[e] - 1, msk = (1 << sh) - 1;
                    const long long wo = wbase + a.lv.woff[e];
                    if constexpr (TWO_D) {
                        const int ox = (bcx & msk) * a.r + kpx, oy = (bcy & msk) * a.r + kpy;
                        const int s = a.lv.size[e];
                        wk = ldf(a.wk, wo + ox, a.w_elems) * ldf(a.wk, wo + s + oy, a.w_elems);
                        wv = ldf(a.wv, wo + ox, a.w_elems) * ldf(a.wv, wo + s + oy, a.w_elems);
                    } else {
                        const int o = (bcx & msk) * a.r + kpx;
                        wk = ldf(a.wk, wo + o, a.w_elems);
                        wv = ldf(a.wv, wo + o, a.w_elems);
                    }
                }
                wkh[j] = static_cast<__bf16>(wk);
                wkl[j] = static_cast<__bf16>(wk - static_cast<float>(wkh[j]));
                wvh[j] = static_cast<__bf16>(wv);
                wvl[j] = static_cast<__bf16>(wv - static_cast<float>(wvh[j]));
            }
#pragma unroll
            for (int db = 0; db < 2; ++db) {
                const int ch = 32 * db + l32;
                const bf16x8 kh = *reinterpret_cast<const bf16x8 *>(ca + ((0 * kHeadDim) + ch) * 16 + 8 * hh);
                const bf16x8 kl = *reinterpret_cast<const bf16x8 *>(ca + ((1 * kHeadDim) + ch) * 16 + 8 * hh);
                const bf16x8 vh = *reinterpret_cast<const bf16x8 *>(ca + ((2 * kHeadDim) + ch) * 16 + 8 * hh);
                const bf16x8 vl = *reinterpret_cast<const bf16x8 *>(ca + ((3 * kHeadDim) + ch) * 16 + 8 * hh);
                f32x16 &dka = db ? dk1 : dk0;
                f32x16 &dva = db ? dv1 : dv0;
                dka = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kh, wkh, dka, 0, 0, 0);
                dka = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kl, wkh, dka, 0, 0, 0);
                dka = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kh, wkl, dka, 0, 0, 0);
                dva = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vh, wvh, dva, 0, 0, 0);
                dva = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vl, wvh, dva, 0, 0, 0);
                dva = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vh, wvl, dva, 0, 0, 0);
            }
            // dots: A rows are the chunk's 16 sets (lanes 16..31 repeat them;
            // those output rows are not stored)
            f32x16 tk = {0}, tv = {0};
            const int m = l32 & 15;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int co = 16 * c + 8 * hh;
                const bf16x8 ah = *reinterpret_cast<const bf16x8 *>(cb + (0 * 16 + m) * PB + co);
                const bf16x8 al = *reinterpret_cast<const bf16x8 *>(cb + (1 * 16 + m) * PB + co);
                const bf16x8 bh = *reinterpret_cast<const bf16x8 *>(cb + (2 * 16 + m) * PB + co);
                const bf16x8 bl = *reinterpret_cast<const bf16x8 *>(cb + (3 * 16 + m) * PB + co);
                tk = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, ko.x[c], tk, 0, 0, 0);
                tk = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, ko.x[c], tk, 0, 0, 0);
                tv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bh, vo.x[c], tv, 0, 0, 0);
                tv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bl, vo.x[c], tv, 0, 0, 0);
            }
            if (klive) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int e = e0 + acc_row(i, hh);   // rows 0..15: this chunk's sets
                    if (e < a.lv.nlev) {
                        const long long di = ((long long)slice * a.lv.nlev + e) * a.n + ktok;
                        stf(a.dotk, di, a.dot_elems, tk[i]);
                        stf(a.dotv, di, a.dot_elems, tv[i]);
                    }
                }
            }
        }
    } else {
        for (int e = 0; e < a.lv.nlev; ++e) {
            const int s = a.lv.size[e];
            __syncthreads();
            if (tid < kHeadDim) {
                long long gb;
                if constexpr (TWO_D)
                    gb = (btok / a.side / s) * a.lv.My[e] + (btok % a.side) / s;
                else
                    gb = btok / s;
                const long long rbase = ((long long)slice * a.R + a.lv.off[e] + gb) * kHeadDim;
                sm.cbar[0][tid] = ldf(a.dkbar, rbase + tid, a.coarse_elems);
                sm.cbar[1][tid] = ldf(a.dvbar, rbase + tid, a.coarse_elems);
            }
            __syncthreads();
            if (!active) continue;
            float wk, wv;
            if constexpr (TWO_D) {
                const long long x = ktok / a.side, y = ktok - (ktok / a.side) * a.side;
                const long long ox = x - (x / s) * s, oy = y - (y / s) * s;
                wk = ldf(a.wk, wbase + a.lv.woff[e] + ox, a.w_elems) * ldf(a.wk, wbase + a.lv.woff[e] + s + oy, a.w_elems);
                wv = ldf(a.wv, wbase + a.lv.woff[e] + ox, a.w_elems) * ldf(a.wv, wbase + a.lv.woff[e] + s + oy, a.w_elems);
            } else {
                wk = ldf(a.wk, wbase + a.lv.woff[e] + (ktok - (ktok / s) * s), a.w_elems);
                wv = ldf(a.wv, wbase + a.lv.woff[e] + (ktok - (ktok / s) * s), a.w_elems);
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int ch = acc_row(i, hh);
                dk0[i] += wk * sm.cbar[0][ch];
                dk1[i] += wk * sm.cbar[0][32 + ch];
                dv0[i] += wv * sm.cbar[1][ch];
                dv1[i] += wv * sm.cbar[1][32 + ch];
            }
            float dkd = 0.f, dvd = 0.f;
#pragma unroll
            for (int c = 0; c < 32; ++c) {
                dkd += ko.x[c] * sm.cbar[0][2 * c + hh];
                dvd += vo.x[c] * sm.cbar[1][2 * c + hh];
            }
            dkd = psum(dkd);
            dvd = psum(dvd);
            if (hh == 0 && klive) {
                const long long di = ((long long)slice * a.lv.nlev + e) * a.n + ktok;
                stf(a.dotk, di, a.dot_elems, dkd);
                stf(a.dotv, di, a.dot_elems, dvd);
            }
        }
    }
    if (!klive) return;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
        const int ch = 8 * g4 + 4 * hh;
        st4<BF16>(a.dk, krow + ch, a.io_elems, dk0[4 * g4], dk0[4 * g4 + 1], dk0[4 * g4 + 2], dk0[4 * g4 + 3]);
        st4<BF16>(a.dk, krow + 32 + ch, a.io_elems, dk1[4 * g4], dk1[4 * g4 + 1], dk1[4 * g4 + 2], dk1[4 * g4 + 3]);
        st4<BF16>(a.dv, krow + ch, a.io_elems, dv0[4 * g4], dv0[4 * g4 + 1], dv0[4 * g4 + 2], dv0[4 * g4 + 3]);
        st4<BF16>(a.dv, krow + 32 + ch, a.io_elems, dv1[4 * g4], dv1[4 * g4 + 1], dv1[4 * g4 + 2], dv1[4 * g4 + 3]);
    }
}

// --------------------------------------------------------------- bwd_weights
// Per (tensor, weight set, weight entry): the dot products of the tokens the
// entry multiplies, over the slices that use the weight set.
//   1D: dpi[o] = sum over groups g of dot[g s + o].
//   2D: Pi = pi_x (x) pi_y, so dpi_x[a] = sum over squares and columns b of
//       pi_y[b] dot[(u s + a) W + v s + b]: the line kernels first form, per pixel
//       row x, T[x] = sum_y pi_y[y mod s] dot[x W + y] and, per column y,
//       U[y] = sum_x pi_x[x mod s] dot[x W + y]; then dpi_x[a] = sum_u T[u s + a]
//       and dpi_y[b] = sum_v U[v s + b].
// Line sums: [2 tensors][S][sets][2 axes][Lm] in `lines`, Lm = max(H, W):
// axis 0 holds the H row sums, axis 1 the W column sums (the rest is unused).

// x + the other lanes' x, the same value in every lane (xor butterfly: each
// lane's order is fixed, so a given lane's result is reproducible)
__device__ inline float wave_sum(float x)
{
#pragma unroll
    for (int sh = 32; sh >= 1; sh >>= 1) x += __shfl_xor(x, sh);
    return x;
}

// Row sums T[x]: 16 lanes per (tensor, slice, set, pixel row), four rows
// per wave; a lane takes four consecutive columns (one 16-byte load) per
// 64 columns, the 16 lanes' sums added by four exchanges (fixed order per
// lane) and stored by the row's first lane.  W is a multiple of 4.
__global__ __launch_bounds__(256) void bwd_row_lines(BwdArgs a, float *lines, long long lines_elems)
{
    const long long rid = (long long)blockIdx.x * 16 + (threadIdx.x >> 4);
    const int l16 = threadIdx.x & 15;
    const int W = a.side, H = a.height, Lm = H > W ? H : W, E = a.lv.nlev;
    const long long total = (long long)a.wsets * a.nslice * E * H;
    const bool live = rid < total;   // the exchanges need every lane
    const long long r = live ? rid : 0;
    const int x = (int)(r % H);
    const int e = (int)((r / H) % E);
    const long long zs = r / ((long long)H * E);   // z * S + slice
    const int z = (int)(zs / a.nslice), slice = (int)(zs - (long long)z * a.nslice);
    const float *dot = z ? a.dotv : a.dotk;
    const float *w = z ? a.wv : a.wk;
    const int s = a.lv.size[e];
    const int hw = a.w_stride ? slice % a.heads : 0;
    const long long wbase = (long long)hw * a.wlen + a.lv.woff[e] + s;   // pi_y
    const long long dbase = ((long long)slice * E + e) * a.n + (long long)x * W;
    float sum = 0.f;
    for (int y = 4 * l16; y < W; y += 64) {
        const uint4 d = ld16(dot, live ? dbase + y : -1, 4, a.dot_elems);
        sum += ldf(w, wbase + y % s, a.w_elems) * __uint_as_float(d.x);
        sum += ldf(w, wbase + (y + 1) % s, a.w_elems) * __uint_as_float(d.y);
        sum += ldf(w, wbase + (y + 2) % s, a.w_elems) * __uint_as_float(d.z);
        sum += ldf(w, wbase + (y + 3) % s, a.w_elems) * __uint_as_float(d.w);
    }
#pragma unroll
    for (int sh = 8; sh >= 1; sh >>= 1) sum += __shfl_xor(sum, sh);
    if (live && l16 == 0) stf(lines, ((zs * E + e) * 2 + 0) * Lm + x, lines_elems, sum);
}

// Column sums U[y]: a workgroup per (tensor, slice, set, 64 consecutive
// pixel columns), lane = column (coalesced); its four waves sum row
// quarters, added in wave order through LDS.
__global__ __launch_bounds__(256) void bwd_col_lines(BwdArgs a, float *lines, long long lines_elems)
{
    __shared__ float red[4][64];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int W = a.side, H = a.height, Lm = H > W ? H : W, E = a.lv.nlev;
    const int cb = (W + 63) / 64;   // column blocks per line set
    const long long gid = blockIdx.x;
    const int yb = (int)(gid % cb);
    const int e = (int)((gid / cb) % E);
    const long long zs = gid / ((long long)cb * E);
    const int z = (int)(zs / a.nslice), slice = (int)(zs - (long long)z * a.nslice);
    const int y = yb * 64 + lane;
    const float *dot = z ? a.dotv : a.dotk;
    const float *w = z ? a.wv : a.wk;
    const int s = a.lv.size[e];
    const int hw = a.w_stride ? slice % a.heads : 0;
    const long long wbase = (long long)hw * a.wlen + a.lv.woff[e];   // pi_x
    const long long dbase = ((long long)slice * E + e) * a.n + y;
    const int x0 = H * wv / 4, x1 = H * (wv + 1) / 4;
    float sum = 0.f;
    if (y < W)
        for (int x = x0; x < x1; ++x) sum += ldf(w, wbase + x % s, a.w_elems) * ldf(dot, dbase + (long long)x * W, a.dot_elems);
    red[wv][lane] = sum;
    __syncthreads();
    if (wv == 0 && y < W)
        stf(lines, ((zs * E + e) * 2 + 1) * Lm + y, lines_elems, (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]));
}

// One wave per (tensor, head's weight set, weight entry): the lanes take the
// (slice of the head, group) terms round-robin, lane 0 stores the butterfly
// sum.  2D sums the line sums of the entry's axis; 1D (blocks that are not a
// multiple of 64) the dot products of the entry's tokens.
template <bool TWO_D>
__global__ __launch_bounds__(256) void bwd_weights(BwdArgs a, const float *lines, long long lines_elems)
{
    const long long wid = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const long long total = (long long)a.wsets * a.heads_w * a.wlen;
    if (wid >= total) return;   // whole waves
    const int z = (int)(wid / ((long long)a.heads_w * a.wlen));
    const long long rem = wid - (long long)z * a.heads_w * a.wlen;
    const int hw = (int)(rem / a.wlen);
    const int wi = (int)(rem - (long long)hw * a.wlen);
    int e = 0;
    while (e + 1 < a.lv.nlev && a.lv.woff[e + 1] <= wi) ++e;
    const int s = a.lv.size[e], E = a.lv.nlev;
    const int o = wi - a.lv.woff[e];
    const float *dot = z ? a.dotv : a.dotk;
    const int nsl = a.w_stride ? a.nslice / a.heads : a.nslice;   // slices that use the weight set
    // 2D: x weights (o < s) sum the row lines, y weights the column lines
    const int axis = TWO_D && o >= s ? 1 : 0;
    const int oo = axis ? o - s : o;
    const int Lm = a.height > a.side ? a.height : a.side;
    const int nl = TWO_D ? (axis ? a.side : a.height) : 0;
    const int ng = TWO_D ? (axis ? a.lv.My[e] : a.lv.M[e]) : a.lv.M[e];
    const long long T = (long long)nsl * ng;
    float sum = 0.f;
    for (long long t = lane; t < T; t += 64) {
        const long long j = t / ng;
        const int u = (int)(t - j * ng);
        const long long sl = a.w_stride ? hw + (long long)a.heads * j : j;
        if constexpr (TWO_D) {
            const long long line = (long long)u * s + oo;
            const long long lbase = ((((long long)z * a.nslice + sl) * E + e) * 2 + axis) * Lm;
            if (line < nl) sum += ldf(lines, lbase + line, lines_elems);
        } else {
            const long long tok = (long long)u * s + o;
            if (tok < a.n) sum += ldf(dot, (sl * E + e) * a.n + tok, a.dot_elems);
        }
    }
    sum = wave_sum(sum);
    if (lane == 0) stf(z ? a.dwv : a.dwk, rem, a.w_elems, sum);
}

// 1D weight gradients, dpi[o] = sum over the slices of the weight set's head
// and the groups g of dot[g s + o]: one workgroup per 64 consecutive entries
// of one set (the sets are 64-entry aligned, r being a multiple of 64).  Its
// eight waves sum disjoint eighths of the (slice, group) terms, sixteen
// loads in flight per lane, and the eighths are added in wave order: a fixed
// order, so results are reproducible.
// Entries [0, 64 nb) of each head (the sets with many terms per entry).
__global__ __launch_bounds__(512) void bwd_weights1d(BwdArgs a, int nb)
{
    constexpr int NWV = 8, NLD = 16;
    __shared__ float red[NWV][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const long long bph = nb;   // 64-entry blocks per head taken here
    const long long id = blockIdx.x;
    const int z = (int)(id / (a.heads_w * bph));
    const long long rem = id - (long long)z * a.heads_w * bph;
    const int hw = (int)(rem / bph);
    const int wi = (int)(rem - (long long)hw * bph) * 64 + lane;
    int e = 0;
    while (e + 1 < a.lv.nlev && a.lv.woff[e + 1] <= wi) ++e;
    const int s = a.lv.size[e], M = a.lv.M[e], E = a.lv.nlev;
    const int o = wi - a.lv.woff[e];
    const float *dot = z ? a.dotv : a.dotk;
    const int nsl = a.w_stride ? a.nslice / a.heads : a.nslice;
    const long long T = (long long)nsl * M;   // terms: slice j of the head, group g
    const long long t0 = T * w / NWV, t1 = T * (w + 1) / NWV;
    long long tj = t0 / M;
    int tg = (int)(t0 - tj * M);
    float acc[NLD];
#pragma unroll
    for (int k = 0; k < NLD; ++k) acc[k] = 0.f;
    for (long long t = t0; t < t1; t += NLD) {
        float v[NLD];
#pragma unroll
        for (int k = 0; k < NLD; ++k) {
            v[k] = 0.f;
            if (t + k < t1) {
                const long long sl = a.w_stride ? hw + (long long)a.heads * tj : tj;
                const long long tok = (long long)tg * s + o;
                if (tok < a.n) v[k] = ldf(dot, (sl * E + e) * a.n + tok, a.dot_elems);
                if (++tg == M) {
                    tg = 0;
                    ++tj;
                }
            }
        }
#pragma unroll
        for (int k = 0; k < NLD; ++k) acc[k] += v[k];
    }
#pragma unroll
    for (int k = NLD / 2; k >= 1; k >>= 1)
#pragma unroll
        for (int i = 0; i < k; ++i) acc[i] += acc[i + k];
    red[w][lane] = acc[0];
    __syncthreads();
    if (w == 0) {
        float tot = red[0][lane];
#pragma unroll
        for (int x = 1; x < NWV; ++x) tot += red[x][lane];
        stf(z ? a.dwv : a.dwk, (long long)hw * a.wlen + wi, a.w_elems, tot);
    }
}

// 1D weight gradients of the sets with fewer than 64 terms per entry (the
// coarse levels, most of the entries): entries [ebeg, wlen) of each head,
// one thread per entry (consecutive entries, coalesced), its terms in
// (slice, group) order with eight loads in flight.
__global__ __launch_bounds__(256) void bwd_weights1d_narrow(BwdArgs a, int ebeg)
{
    const long long nent = a.wlen - ebeg;
    const long long id = (long long)blockIdx.x * 256 + threadIdx.x;
    if (id >= (long long)a.wsets * a.heads_w * nent) return;
    const int z = (int)(id / (a.heads_w * nent));
    const long long rem = id - (long long)z * a.heads_w * nent;
    const int hw = (int)(rem / nent);
    const int wi = ebeg + (int)(rem - (long long)hw * nent);
    int e = 0;
    while (e + 1 < a.lv.nlev && a.lv.woff[e + 1] <= wi) ++e;
    const int s = a.lv.size[e], M = a.lv.M[e], E = a.lv.nlev;
    const int o = wi - a.lv.woff[e];
    const float *dot = z ? a.dotv : a.dotk;
    const int nsl = a.w_stride ? a.nslice / a.heads : a.nslice;
    const int T = nsl * M;   // terms: slice j of the head, group g
    int tj = 0, tg = 0;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int t = 0; t < T; t += 8) {
        float v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            v[k] = 0.f;
            if (t + k < T) {
                const long long sl = a.w_stride ? hw + (long long)a.heads * tj : tj;
                const long long tok = (long long)tg * s + o;
                if (tok < a.n) v[k] = ldf(dot, (sl * E + e) * a.n + tok, a.dot_elems);
                if (++tg == M) {
                    tg = 0;
                    ++tj;
                }
            }
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[k] += v[k];
    }
    stf(z ? a.dwv : a.dwk, (long long)hw * a.wlen + wi, a.w_elems,
        ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7])));
}

// dpi of one weight tensor from its dot products (a.dotk, a.wk -> a.dwk when
// a.wsets == 1; both tensors when it is 2)
template <bool TWO_D>
hipError_t launch_weights(const BwdArgs &a, hipStream_t st)
{
    hipError_t e = hipSuccess;
    // the 2D line sums reuse the partials' space, free after bwd_reduce
    float *lines = a.part;
    long long lines_elems = 0;
    if constexpr (TWO_D) {
        lines_elems = (long long)a.wsets * a.nslice * a.lv.nlev * 2 * (a.height > a.side ? a.height : a.side);
        if (lines_elems > a.part_elems) return hipErrorInvalidValue;
        const long long rows = (long long)a.wsets * a.nslice * a.lv.nlev * a.height;   // 16 lanes each
        const long long colb = (long long)a.wsets * a.nslice * a.lv.nlev * ((a.side + 63) / 64);
        if (a.side % 4) return hipErrorInvalidValue;
        hipLaunchKernelGGL(bwd_row_lines, dim3((unsigned)((rows + 15) / 16)), dim3(256), 0, st, a, lines, lines_elems);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(bwd_col_lines, dim3((unsigned)colb), dim3(256), 0, st, a, lines, lines_elems);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const long long nw = (long long)a.wsets * a.heads_w * a.wlen;
    if (TWO_D || a.r % 64)   // 1D sets are 64-entry aligned when r is a multiple of 64
        hipLaunchKernelGGL((bwd_weights<TWO_D>), dim3((unsigned)((nw + 3) / 4)), dim3(256), 0, st, a, lines,
                           lines_elems);
    else {
        // sets with at least 64 terms per entry: a workgroup per 64 entries;
        // the rest (a suffix of the sets: terms shrink with the level): a
        // thread per entry
        const int nsl = a.w_stride ? a.nslice / a.heads : a.nslice;
        int es = 0;
        while (es < a.lv.nlev && (long long)nsl * a.lv.M[es] >= 64) ++es;
        const int ebeg = es < a.lv.nlev ? a.lv.woff[es] : a.wlen;
        if (ebeg % 64) return hipErrorInvalidValue;
        if (ebeg > 0) {
            hipLaunchKernelGGL(bwd_weights1d, dim3((unsigned)((long long)a.wsets * a.heads_w * (ebeg / 64))), dim3(512),
                               0, st, a, ebeg / 64);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        const long long nn = (long long)a.wsets * a.heads_w * (a.wlen - ebeg);
        if (nn > 0) hipLaunchKernelGGL(bwd_weights1d_narrow, dim3((unsigned)((nn + 255) / 256)), dim3(256), 0, st, a, ebeg);
    }
    return hipGetLastError();
}

template <bool BF16, bool TWO_D, int NW, bool PL, bool LIN>
hipError_t launch_all(const BwdArgs &a0, hipStream_t st)
{
    BwdArgs a = a0;
    const int cpb = (a.qtile + 31) / 32;   // 32-query chunks per block (a block below 32 is one)
    a.npart = a.nblocks * ((cpb + NW - 1) / NW);   // (query block, workgroup) rows per slice
    if (a.pslices <= 0) return hipErrorInvalidValue;
    if ((long long)2 * a.pslices * a.npart * a.nslot * kHeadDim > a.part_elems && a.lv.nlev > 0)
        return hipErrorInvalidValue;
    if (LIN && a.lv.nlev > 0 &&
        ((long long)a.nslice * a.npart * a.lv.nlev * kHeadDim > a.qpart_elems ||
         (long long)a.nslice * a.n * kHeadDim > a.dqn_elems || a.lv.nlev > kMaxCoarse))
        return hipErrorInvalidValue;
    // FMA-linear dq: workgroups of 32 tokens, 32-bit token and workgroup indices
    const long long runs_ll = (a.n + 31) / 32;
    if (LIN && (a.n > 0x7fffffffLL - 32 || (long long)a.nslice * runs_ll > 0x7fffffffLL)) return hipErrorInvalidValue;
    const int runs = (int)runs_ll;
    hipError_t e = hipSuccess;
    const long long per_slice = (long long)a.nblocks * ((cpb + NW - 1) / NW);   // query-pass workgroups
    // the query pass and the reduction of its partials, pslices slices at a time
    for (int s0 = 0; s0 < a.nslice; s0 += a.pslices) {
        BwdArgs b = a;
        b.slice0 = s0;
        const int cnt = a.nslice - s0 < a.pslices ? a.nslice - s0 : a.pslices;
        hipLaunchKernelGGL((bwd_query<BF16, TWO_D, NW, PL, LIN>), dim3((unsigned)(cnt * per_slice)), dim3(64 * NW), 0,
                           st, b);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (a.lv.nlev > 0) {
            // grid over [2][pslices][R]; the rows of slices past the last one return at once
            const long long nr = 2LL * a.pslices * a.R;
            hipLaunchKernelGGL((bwd_reduce<TWO_D>), dim3((unsigned)nr), dim3(64), 0, st, b);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
    }
    const unsigned groups = (unsigned)((long long)a.nslice * per_slice);
    hipLaunchKernelGGL((bwd_key<BF16, TWO_D, NW>), dim3(groups), dim3(64 * NW), 0, st, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (a.lv.nlev > 0) {
        BwdArgs w = a;
        w.wsets = 2;
        if ((e = launch_weights<TWO_D>(w, st)) != hipSuccess) return e;
        if constexpr (LIN) {
            // dQ_bar, then dq and q_t . dQ_bar, then dpi^q
            hipLaunchKernelGGL((bwd_qreduce<TWO_D>), dim3((unsigned)((long long)a.nslice * a.R)), dim3(64), 0, st,
                               a);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            hipLaunchKernelGGL((bwd_qapply<BF16, TWO_D>), dim3((unsigned)((long long)a.nslice * runs)), dim3(256), 0,
                               st, a, runs);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            BwdArgs wq = a;
            wq.wsets = 1;
            wq.dotk = a.dotq;
            wq.wk = a.wq;
            wq.dwk = a.dwq;
            if ((e = launch_weights<TWO_D>(wq, st)) != hipSuccess) return e;
        }
    } else if constexpr (LIN) {
        // no coarse level: dq is the near field's part
        hipLaunchKernelGGL((bwd_qapply<BF16, TWO_D>), dim3((unsigned)((long long)a.nslice * runs)), dim3(256), 0, st,
                           a, runs);
        e = hipGetLastError();
    }
    return e;
}

// Waves per workgroup: four for bf16 blocks of 4 or 8 chunks (128 or 256
// tokens), else two (fp32 keeps two: its LDS tiles are twice as large).
// The plan sizes the coarse partials (one row per block and workgroup) with
// the same rule.
template <bool BF16, bool TWO_D, bool PL, bool LIN>
hipError_t launch_nw(const BwdArgs &a, hipStream_t st)
{
    if constexpr (BF16)
        if (a.qtile % 128 == 0) return launch_all<BF16, TWO_D, 4, PL, LIN>(a, st);
    return launch_all<BF16, TWO_D, 2, PL, LIN>(a, st);
}

template <bool BF16, bool TWO_D>
hipError_t launch_norm(const BwdArgs &a, hipStream_t st)
{
    if (a.norm_level) {
        // a level must be one aligned group of a 32-slot block
        if (a.slot_group != 4 && a.slot_group != 8 && a.slot_group != 16 && a.slot_group % 32)
            return hipErrorInvalidValue;
        if (a.nslot > a.slot_group * kMaxCoarse) return hipErrorInvalidValue;
        if (a.qbar) return hipErrorInvalidValue;
        return launch_nw<BF16, TWO_D, true, false>(a, st);
    }
    if (a.qbar) return launch_nw<BF16, TWO_D, false, true>(a, st);   // FMA-linear
    return launch_nw<BF16, TWO_D, false, false>(a, st);
}

}  // namespace

hipError_t launch_backward(const BwdArgs &a, bool bf16, bool two_d, hipStream_t st)
{
    if (a.nslice == 0 || a.n == 0) return hipSuccess;
    if (bf16) return two_d ? launch_norm<true, true>(a, st) : launch_norm<true, false>(a, st);
    return two_d ? launch_norm<false, true>(a, st) : launch_norm<false, false>(a, st);
}

}  // namespace fma_dev
