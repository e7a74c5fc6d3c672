// coarsen.hip -- per-level coarse keys/values (Eq. agg1d, Eq. agg2d) on gfx950.
//
// Every level is built straight from the fine tokens, so K and V are read
// from HBM exactly once.  Four kernels:
//   coarsen1d_stream  (1D, bf16) and coarsen2d_stream (2D, bf16): the level
//                     sums on the matrix cores, every wave an independent
//                     streamer of units (CW tokens in 1D, 32x32-pixel tiles
//                     in 2D; see the comments above the kernels);
//   coarsen1d_chunks  (1D, fp32) and coarsen2d_tiles (2D, fp32, and bf16 maps
//                     the streaming kernel does not take): a workgroup owns a
//                     chunk of CH consecutive tokens (1D) or a 32x32 tile of
//                     the token map (2D) of one (batch, head, tensor); each
//                     thread streams a "run" of rows for 8 channels (16-byte
//                     loads, eight threads cover one 128-byte row) and keeps
//                     one fp32 partial sum per level and channel in registers;
//                     a run never crosses a base block, so it lies in exactly
//                     one group of every level, and the runs of a group are
//                     summed in LDS in a fixed order.
// Levels whose groups are wider than a unit / chunk / tile leave one fp32
// partial per unit, and coarsen_finish adds the partials of each group in
// ascending order: no atomics, bitwise reproducible.
#include <string.h>

#include "fma_device.hpp"
#include "fma_kernels.hpp"

namespace fma_dev {

namespace {

// 8 consecutive channels of one row as fp32.
template <bool BF16>
__device__ inline void load8(const void *base, long long elem, float (&x)[8])
{
    if constexpr (BF16) {
        const uint4 w = *reinterpret_cast<const uint4 *>(static_cast<const __bf16 *>(base) + elem);
        x[0] = bf16lo_to_f32(w.x); x[1] = bf16hi_to_f32(w.x);
        x[2] = bf16lo_to_f32(w.y); x[3] = bf16hi_to_f32(w.y);
        x[4] = bf16lo_to_f32(w.z); x[5] = bf16hi_to_f32(w.z);
        x[6] = bf16lo_to_f32(w.w); x[7] = bf16hi_to_f32(w.w);
    } else {
        const float4 *p = reinterpret_cast<const float4 *>(static_cast<const float *>(base) + elem);
        const float4 u = p[0], w = p[1];
        x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
        x[4] = w.x; x[5] = w.y; x[6] = w.z; x[7] = w.w;
    }
}

// Raw 8-channel row piece as loaded (16 bytes of bf16 or 32 bytes of fp32),
// so loads can be issued ahead of the arithmetic that consumes them.
template <bool BF16>
struct Raw8;
template <>
struct Raw8<true> {
    uint4 w;
};
template <>
struct Raw8<false> {
    float4 a, b;
};

template <bool BF16>
__device__ inline Raw8<BF16> load_raw(const void *base, long long elem)
{
    Raw8<BF16> r;
    if constexpr (BF16) {
        r.w = *reinterpret_cast<const uint4 *>(static_cast<const __bf16 *>(base) + elem);
    } else {
        const float4 *p = reinterpret_cast<const float4 *>(static_cast<const float *>(base) + elem);
        r.a = p[0];
        r.b = p[1];
    }
    return r;
}

template <bool BF16>
__device__ inline Raw8<BF16> zero_raw()
{
    Raw8<BF16> r;
    if constexpr (BF16)
        r.w = make_uint4(0, 0, 0, 0);
    else
        r.a = r.b = make_float4(0.f, 0.f, 0.f, 0.f);
    return r;
}

template <bool BF16>
__device__ inline void unpack8(const Raw8<BF16> &r, float (&x)[8])
{
    if constexpr (BF16) {
        x[0] = bf16lo_to_f32(r.w.x); x[1] = bf16hi_to_f32(r.w.x);
        x[2] = bf16lo_to_f32(r.w.y); x[3] = bf16hi_to_f32(r.w.y);
        x[4] = bf16lo_to_f32(r.w.z); x[5] = bf16hi_to_f32(r.w.z);
        x[6] = bf16lo_to_f32(r.w.w); x[7] = bf16hi_to_f32(r.w.w);
    } else {
        x[0] = r.a.x; x[1] = r.a.y; x[2] = r.a.z; x[3] = r.a.w;
        x[4] = r.b.x; x[5] = r.b.y; x[6] = r.b.z; x[7] = r.b.w;
    }
}

template <bool BF16>
__device__ inline void store1(void *base, long long elem, float v)
{
    if constexpr (BF16)
        static_cast<uint16_t *>(base)[elem] = static_cast<uint16_t>(f32_to_bf16_bits(v));
    else
        static_cast<float *>(base)[elem] = v;
}

}  // namespace

// ---------------------------------------------------------------- 1D
// grid (nchunk, nslice, 2): blockIdx.z selects K (0) or V (1).  A thread
// takes 8 of the D channels over a run of RUN rows: D / 8 threads per row,
// NRUN = 2048 / D runs of a chunk (CH = NRUN * RUN).
template <bool BF16, int NLEV, int D>
__global__ __launch_bounds__(256) void coarsen1d_chunks(CoarsenArgs a)
{
    extern __shared__ __attribute__((aligned(16))) float smem[];
    constexpr int CPR = D / 8, NRUN = 256 / CPR;
    const int chunk = blockIdx.x, slice = blockIdx.y, z = blockIdx.z;
    const int tid = threadIdx.x, c8 = tid % CPR, run = tid / CPR;
    const int CH = a.chunk, RUN = a.run;
    const long long n = a.n;
    const float *pi = (z ? a.wv : a.wk) + (long long)(slice % a.heads) * a.w_stride;

    // Weight windows: level l needs pi_l[(chunk*CH) mod s_l + t], t < min(s_l, CH).
    int wlo[NLEV], wlen[NLEV];
    int wtot = 0;
#pragma unroll
    for (int l = 0; l < NLEV; ++l) {
        const int s = a.lv.size[l];
        wlen[l] = s < CH ? s : CH;
        wlo[l] = wtot;
        const long long start = s > CH ? ((long long)chunk * CH) % s : 0;
        for (int t = tid; t < wlen[l]; t += 256) smem[wtot + t] = pi[a.lv.woff[l] + start + t];
        wtot += wlen[l];
    }
    float *red = smem + wtot;   // [2][NRUN runs][D channels]
    __syncthreads();

    const long long row0 = (long long)chunk * CH + (long long)run * RUN;
    const void *src = z ? a.v : a.k;
    const long long sbase = (long long)slice * n * D + c8 * 8;

    float acc[NLEV][8];
#pragma unroll
    for (int l = 0; l < NLEV; ++l)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[l][c] = 0.f;

    int wb[NLEV];
#pragma unroll
    for (int l = 0; l < NLEV; ++l) wb[l] = wlo[l] + (run * RUN) % wlen[l];

    // rows are loaded four at a time, one group ahead of the arithmetic
    Raw8<BF16> cur[4], nxt[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const long long row = row0 + u;
        cur[u] = row < n ? load_raw<BF16>(src, sbase + row * D) : zero_raw<BF16>();
    }
    for (int rr = 0; rr < RUN; rr += 4) {
        if (rr + 4 < RUN) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const long long row = row0 + rr + 4 + u;
                nxt[u] = row < n ? load_raw<BF16>(src, sbase + row * D) : zero_raw<BF16>();
            }
        }
        float xv[4][8];
#pragma unroll
        for (int u = 0; u < 4; ++u) unpack8<BF16>(cur[u], xv[u]);
#pragma unroll
        for (int l = 0; l < NLEV; ++l) {
            // weights of rows rr .. rr+3 (16-byte aligned: window bases and run
            // offsets are multiples of 4 floats)
            const float4 w4 = *reinterpret_cast<const float4 *>(&smem[wb[l] + rr]);
            const float w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int c = 0; c < 8; ++c) acc[l][c] = fmaf(w[u], xv[u][c], acc[l][c]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) cur[u] = nxt[u];
    }

    const int zs = z * a.nslice + slice;
    void *kbar = a.coarse;
#pragma unroll
    for (int l = 0; l < NLEV; ++l) {
        float *buf = red + (l & 1) * NRUN * D;
        *reinterpret_cast<float4 *>(&buf[run * D + c8 * 8]) =
            make_float4(acc[l][0], acc[l][1], acc[l][2], acc[l][3]);
        *reinterpret_cast<float4 *>(&buf[run * D + c8 * 8 + 4]) =
            make_float4(acc[l][4], acc[l][5], acc[l][6], acc[l][7]);
        __syncthreads();
        const int s = a.lv.size[l];
        if (s <= CH) {
            const int G = CH / s, rpg = s / RUN;
            for (int o = tid; o < G * D; o += 256) {
                const int g = o / D, c = o - g * D;
                float sum = 0.f;
                for (int t = 0; t < rpg; ++t) sum += buf[(g * rpg + t) * D + c];
                const long long m = (long long)chunk * G + g;
                if (m < a.lv.M[l])
                    store1<BF16>(kbar, ((long long)zs * a.R + a.lv.off[l] + m) * D + c, sum);
            }
        } else if (tid < D) {
            float sum = 0.f;
            for (int t = 0; t < NRUN; ++t) sum += buf[t * D + tid];
            const long long pl = l - a.first_partial;
            a.part[(((long long)zs * a.npartial + pl) * a.part_count + chunk) * D + tid] = sum;
        }
    }
}

// bf16 1D coarsening on the matrix cores.
//
// For the tokens of one 16-row step the sums of every level are a single
// contraction,
//     Dacc[c][col] += sum_k K[t0 + k][c] * Wt[k][col],   c < 64, col < 32,
// where column col = part * 16 + level holds, for part 0, the bf16 rounding
// hi of the level's fp32 weight and, for part 1, the bf16 rounding of the
// remainder w - hi (split in registers at each step).  hi + lo represents the
// weight to about 2^-17 relative, so the bf16 products summed in fp32 keep the
// fp32 weights' accuracy; the two parts of a level are added when its group
// is written out.  Each step is two v_mfma_f32_32x32x16_bf16 (channels 0-31
// and 32-63) with A = K^T, read from a row-major LDS tile with the
// transposing ds_read_b64_tr_b16, and B = the step's 16 x 32 weight slice.
// With all levels on the matrix cores the per-element arithmetic no longer
// limits the pass: it streams K and V once.
//
// Work split.  Every wave is an independent streamer.  The (tensor, slice)
// rows are cut into units of CW tokens (CW = r * 2^k); wave g takes units
// g, g + G, g + 2G, ... (G waves in the grid, sized so that every wave gets
// the same number of units up to one).  A unit's steps flow through the
// wave's ring of D slots with direct-to-LDS loads issued D steps ahead, across
// unit boundaries, so the stream never drains.  A slot holds the step's 16
// K (or V) rows and the 16 weights of each level for those rows, gathered
// from the weight vectors by the same loads.  Groups no wider than CW close
// inside a unit and are written out as they close; each unit leaves one fp32
// sum for every wider group it lies in, which coarsen_finish adds in
// ascending unit order.  No barrier, no atomics.
//
// Tile layout and operand orders follow the fused attention kernel's V tile:
// chunk c of row r sits at chunk position c ^ (2 * (r & 3)), and the
// transposing read hands lane i (h = i / 32) the rows
// {4h .. 4h+3, 8+4h .. 8+4h+3} of the step as its eight k-slots, so the lane
// takes the weights of those rows (two aligned 16-byte reads).
__device__ inline void dma16_row(const void *gptr, uint32_t lds_base)
{
    asm volatile("global_load_lds_dwordx4 %0, off" : : "v"(gptr), "{m0}"(lds_base) : "memory");
}

// Scalar-base forms: address = sbase + voff (32-bit per-lane offset).  No
// immediate offset is used: on these loads it would move the LDS destination
// as well.  The K / V rows are read once per pass: their loads are streaming
// (non-temporal), which measured 8-15 % faster; the weights, read by every
// unit of a head, keep the default policy.
__device__ inline void dma16_sv(uint32_t voff, const void *sbase, uint32_t lds_base)
{
    asm volatile("global_load_lds_dwordx4 %0, %1 nt" : : "v"(voff), "s"(sbase), "{m0}"(lds_base) : "memory");
}

__device__ inline void dma4_sv(uint32_t voff, const void *sbase, uint32_t lds_base)
{
    asm volatile("global_load_lds_dword %0, %1" : : "v"(voff), "s"(sbase), "{m0}"(lds_base) : "memory");
}

template <int N>
__device__ inline void wait_vm()
{
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ inline void wait_lgkm0()
{
    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

// Wait until the loads of the oldest step in flight have landed.  With the
// ring full, D - 1 later steps (NLD loads each) may stay in flight; near the
// end of the stream everything is drained.  Later stores only make the wait
// longer: the counter retires in issue order.
template <int NLD, int D>
__device__ inline void wait_oldest(bool full)
{
    static_assert(NLD * (D - 1) < 64, "vmcnt range");
    if (full)
        wait_vm<NLD * (D - 1)>();
    else
        wait_vm<0>();
}

// two fp32 -> packed bf16, round to nearest even (v_cvt_pk_bf16_f32)
__device__ inline uint32_t cvt_pk_bf16(float lo, float hi)
{
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 p = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
    return __builtin_bit_cast(uint32_t, p);
}

typedef short s16x4c __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4c lds_s16x4c;

// The hi / lo bf16 halves of a lane's eight fp32 weights (part 0 lanes take
// the bf16 rounding, part 1 lanes the remainder) as the B operand.
__device__ inline bf16x8 split_weights(const f32x4 &w0, const f32x4 &w1, int pt)
{
    const float wv8[8] = {w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
    uint32_t bp[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const uint32_t hb = cvt_pk_bf16(wv8[2 * e], wv8[2 * e + 1]);
        const uint32_t lb = cvt_pk_bf16(wv8[2 * e] - bf16lo_to_f32(hb), wv8[2 * e + 1] - bf16hi_to_f32(hb));
        bp[e] = pt ? lb : hb;
    }
    typedef uint32_t u32x4c __attribute__((ext_vector_type(4)));
    return __builtin_bit_cast(bf16x8, (u32x4c{bp[0], bp[1], bp[2], bp[3]}));
}

// Fold the hi and lo columns of a pair of accumulators (channels 0..31 and
// 32..63 of every set), four values at a time: v_permlane16_swap exchanges
// the odd 16-lane rows of its first operand with the even rows of its
// second, so one swap and one add leave each part-0 lane with hi + lo of
// channels 0..31 and each part-1 lane with hi + lo of channels 32..63.
// Values jj * 4 .. jj * 4 + 3 of a lane are then channels
// 32 pt + 8 jj + 4 h + 0..3 of its set.
__device__ inline f32x4 fold_parts4(const f32x16 &c0, const f32x16 &c1, int jj)
{
    f32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int j = 4 * jj + i;
        const auto sw = __builtin_amdgcn_permlane16_swap(__float_as_uint(c0[j]), __float_as_uint(c1[j]), false, false);
        r[i] = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
    }
    return r;
}

// One wave per unit of CW consecutive tokens of one (tensor, slice), a ring
// of D slots of 16 tokens each filled by direct-to-LDS loads.  Every 16-token
// step is one 32x32x16 matrix-core product per 32 channels and per group of
// 16 coarse sets: A = the 16 rows transposed (channels x tokens), B = the
// rows' weights of each set, split into bf16 hi and lo columns, so that every
// accumulator column holds one set's running sum (hi or lo part) in fp32.
// NWD weight loads of four sets each fill a slot; with more than 16 sets
// (NWD > 4) a second column group covers sets 16 .. 31.
template <int D, int NWD>
__global__ __launch_bounds__(256) void coarsen1d_stream(CoarsenArgs a)
{
    extern __shared__ __attribute__((aligned(16))) unsigned char csm[];
    static_assert(D >= 2 && D <= 6 && NWD >= 1 && NWD <= 8, "ring shape");
    constexpr int CG = NWD > 4 ? 2 : 1;      // column groups of 16 sets
    constexpr int DATAB = 16 * 128;          // 16 bf16 rows
    constexpr int SLOTB = DATAB + 256 * NWD; // + 16 weights of up to 4 * NWD sets
    constexpr int NLD = 2 + NWD;             // loads per step
    // the host sizes each wave's LDS with the same formula; a launch that
    // does not match it does nothing
    if (a.wave_lds < stream_wave_lds(D, NWD) || a.lv.nlev > 4 * NWD) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // per wave: D slots | 64 zero bytes | 16 staged bf16 output rows | their
    // 16 row indices (-1: a group past the end of the sequence)
    unsigned char *const ring = csm + wave * a.wave_lds;
    unsigned char *const zero = ring + D * SLOTB;
    __bf16 *const orow = reinterpret_cast<__bf16 *>(zero + 64);                  // [16][64]
    int *const odst = reinterpret_cast<int *>(zero + 64 + 2048);                 // [16]
    if (lane < 16) reinterpret_cast<float *>(zero)[lane] = 0.f;
    const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(
        static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void *)ring)));

    const int CW = a.chunk, nsteps = CW >> 4, nlev = a.lv.nlev;
    const long long n = a.n;
    const int upz = a.nchunk;                          // units per (tensor, slice)
    const int U = 2 * a.nslice * upz;
    const int G = gridDim.x * 4;
    const int gw = blockIdx.x * 4 + wave;
    int ndir = 0;
    while (ndir < nlev && a.lv.size[ndir] <= CW) ++ndir;

    // ---- issue side: lane L of weight load i gathers weight L % 16 of set 4 i + L / 16
    // units and groups are both r times powers of two wide: a unit starts at
    // position (c mod wsz / CW) * CW of a group wider than CW, at 0 otherwise
    int wsz[NWD], wof[NWD], wmask[NWD];
#pragma unroll
    for (int i = 0; i < NWD; ++i) {
        // lanes of sets past the last one read weight 0 of the first set, every step
        const int lvl = 4 * i + (lane >> 4);
        wsz[i] = 16;
        wof[i] = 0;
        if (lvl < nlev) {   // one indexed read of the set table per lane
            wsz[i] = a.lv.size[lvl];
            wof[i] = a.lv.woff[lvl] + (lane & 15);
        }
        wmask[i] = wsz[i] > a.chunk ? wsz[i] / a.chunk - 1 : 0;
    }
    const uint32_t rowoff = (lane >> 3) * 128 + 16 * ((lane & 7) ^ (2 * ((lane >> 3) & 3)));
    const uint32_t rowoff8 = rowoff + 1024;   // rows 8 .. 15 of the step
    int iu = gw, ist = 0, inv = 0, islot = 0;
    const char *isrc = nullptr;      // first row of the step to issue (uniform)
    const float *ipi = nullptr;      // weight vectors of the unit's head (uniform)
    int ipos[NWD];                   // position of the step's first token in each lane's set group
#define FMA_UNIT_ISSUE_SETUP()                                                                          \
    do {                                                                                                \
        const int zs_ = iu / upz, c_ = iu - zs_ * upz;                                                  \
        const int z_ = zs_ >= a.nslice, sl_ = zs_ - z_ * a.nslice;                                      \
        const long long t0_ = (long long)c_ * CW;                                                       \
        const long long left_ = (n - t0_) >> 4;                                                         \
        inv = left_ < nsteps ? (int)left_ : nsteps;                                                     \
        isrc = static_cast<const char *>(z_ ? a.v : a.k) + ((long long)sl_ * n + t0_) * 128;            \
        ipi = (z_ ? a.wv : a.wk) + (long long)(sl_ % a.heads) * a.w_stride;                             \
        for (int i_ = 0; i_ < NWD; ++i_) ipos[i_] = (c_ & wmask[i_]) * CW;                              \
    } while (0)
    if (iu < U) FMA_UNIT_ISSUE_SETUP();
    int issued = 0;   // steps issued, counted since the start
    auto issue_next = [&]() {
        if (iu >= U) return;
        const uint32_t dst = ring_lds + islot * SLOTB;
        dma16_sv(rowoff, isrc, dst);
        dma16_sv(rowoff8, isrc, dst + 1024);
#pragma unroll
        for (int i = 0; i < NWD; ++i) {
            dma4_sv(4u * (uint32_t)(wof[i] + ipos[i]), ipi, dst + DATAB + 256 * i);
            ipos[i] += 16;
            ipos[i] = ipos[i] >= wsz[i] ? ipos[i] - wsz[i] : ipos[i];
        }
        ++issued;
        isrc += DATAB;
        islot = islot + 1 == D ? 0 : islot + 1;
        if (++ist == inv) {
            ist = 0;
            iu += G;
            if (iu < U) FMA_UNIT_ISSUE_SETUP();
        }
    };
#undef FMA_UNIT_ISSUE_SETUP

    // ---- consume side: accumulator column c of group g holds set 16 g + c % 16, part c / 16
    const int col = lane & 31, lv_ = col & 15, pt = col >> 4, h = lane >> 5;
    // this lane's weights in a slot; columns past the last set read zeros
    const bool on0 = lv_ < nlev, on1 = CG == 2 && 16 + lv_ < nlev;
    const int wread0 = DATAB + 64 * (on0 ? lv_ : 0) + 16 * h;
    const int wread1 = DATAB + 64 * (on1 ? 16 + lv_ : 0) + 16 * h;
    int voff[2];
    {
        const int gq = lane >> 4, s4 = lane & 15, j = s4 >> 2, q = s4 & 3;
        const int row = 4 * (gq >> 1) + j;
#pragma unroll
        for (int db = 0; db < 2; ++db) {
            const int ch = 4 * db + 2 * (gq & 1) + (q >> 1);
            voff[db] = row * 128 + 16 * (ch ^ (2 * (row & 3))) + 8 * (q & 1);
        }
    }
    const int first16 = ndir > 0 ? a.lv.size[0] >> 4 : 1 << 30;   // steps per narrowest group
    // a set's groups are 2^(its level - the narrowest set's level) narrowest
    // groups wide, and a unit 2^cwsh of them
    const int lvl0 = a.lv.lvl[0];
    int cwsh = 0;
    while (ndir > 0 && (a.lv.size[0] << cwsh) < CW) ++cwsh;
    // the lane's set in each column group: its width exponent, groups, first row
    int se[CG], sM[CG], soff[CG];
#pragma unroll
    for (int g = 0; g < CG; ++g) {
        const int l = 16 * g + lv_;
        se[g] = 0;
        sM[g] = 0;
        soff[g] = 0;
        if (l < nlev) {
            se[g] = a.lv.lvl[l] - lvl0;
            sM[g] = a.lv.M[l];
            soff[g] = a.lv.off[l];
        }
    }

#pragma unroll
    for (int j = 0; j < D; ++j) issue_next();

    int consumed = 0, cslot = 0, nout = 0;
    // write the staged bf16 rows (8 per store instruction) and empty the staging
#define FMA_FLUSH_ROWS()                                                                                  \
    do {                                                                                                  \
        for (int k0 = 0; k0 < nout; k0 += 8) {                                                            \
            const int k = k0 + (lane >> 3);                                                               \
            const uint4 v = *reinterpret_cast<const uint4 *>(orow + k * 64 + 8 * (lane & 7));             \
            const int dk = odst[k];                                                                       \
            if (k < nout && dk >= 0)                                                                      \
                *reinterpret_cast<uint4 *>(static_cast<__bf16 *>(a.coarse) + (long long)dk * kHeadDim +     \
                                           8 * (lane & 7)) = v;                                           \
        }                                                                                                 \
        nout = 0;                                                                                         \
    } while (0)
    f32x16 acc0 = {0}, acc1 = {0}, acc2 = {0}, acc3 = {0};
    for (int cu = gw; cu < U; cu += G) {
        const int zs = cu / upz, c = cu - zs * upz;
        const long long t0 = (long long)c * CW;
        const long long leftc = (n - t0) >> 4;
        const int nv = leftc < nsteps ? (int)leftc : nsteps;
        int left0 = first16;
        int kk = 0;   // narrowest groups closed so far in this unit
        for (int st = 0; st < nsteps; ++st) {
            if (st < nv) {
                wait_oldest<NLD, D>(issued - consumed == D);
                const unsigned char *sl = ring + cslot * SLOTB;
                bf16x8 av[2];
#pragma unroll
                for (int db = 0; db < 2; ++db) {
                    const s16x4c r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4c *)(sl + voff[db]));
                    const s16x4c r2 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4c *)(sl + 8 * 128 + voff[db]));
                    typedef short s16x8 __attribute__((ext_vector_type(8)));
                    const s16x8 t = {r1[0], r1[1], r1[2], r1[3], r2[0], r2[1], r2[2], r2[3]};
                    av[db] = __builtin_bit_cast(bf16x8, t);
                }
                // weights of the lane's k-slots (rows 4h .. 4h+3 and 8+4h .. 8+4h+3)
                const unsigned char *wp0 = on0 ? sl + wread0 : zero;
                const f32x4 w00 = *reinterpret_cast<const f32x4 *>(wp0);
                const f32x4 w01 = *reinterpret_cast<const f32x4 *>(wp0 + 32);
                f32x4 w10 = {0.f, 0.f, 0.f, 0.f}, w11 = {0.f, 0.f, 0.f, 0.f};
                if constexpr (CG == 2) {
                    const unsigned char *wp1 = on1 ? sl + wread1 : zero;
                    w10 = *reinterpret_cast<const f32x4 *>(wp1);
                    w11 = *reinterpret_cast<const f32x4 *>(wp1 + 32);
                }
                wait_lgkm0();   // the slot is read: refill it
                ++consumed;
                cslot = cslot + 1 == D ? 0 : cslot + 1;
                issue_next();
                const bf16x8 bw0 = split_weights(w00, w01, pt);
                acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[0], bw0, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[1], bw0, acc1, 0, 0, 0);
                if constexpr (CG == 2) {
                    const bf16x8 bw1 = split_weights(w10, w11, pt);
                    acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[0], bw1, acc2, 0, 0, 0);
                    acc3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[1], bw1, acc3, 0, 0, 0);
                }
            }
            // groups that close at the end of this step: those of a prefix of
            // the sets (a wider set can only close where the narrower ones do;
            // units start on a boundary of every set below ndir), folded and
            // staged together, up to 16 sets of one column group at a time
            if (--left0 > 0) continue;
            left0 = first16;
            ++kk;
            int lc = 0;
            while (lc < ndir && !(kk & ((1 << (a.lv.lvl[lc] - lvl0)) - 1))) ++lc;
#pragma unroll
            for (int g = 0; g < CG; ++g) {
                const int cn = lc - 16 * g < 16 ? lc - 16 * g : 16;   // closing sets of this group
                if (cn <= 0) break;
                if (nout + cn > 16) FMA_FLUSH_ROWS();
                __bf16 *const dst = orow + (nout + (lv_ < cn ? lv_ : 0)) * 64 + 32 * pt + 4 * h;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const f32x4 f = g ? fold_parts4(acc2, acc3, jj) : fold_parts4(acc0, acc1, jj);
                    if (lv_ < cn) *reinterpret_cast<uint2 *>(dst + 8 * jj) = uint2{cvt_pk_bf16(f[0], f[1]), cvt_pk_bf16(f[2], f[3])};
                }
                if (lv_ < cn) {
                    if (pt == 0 && h == 0) {
                        const long long m = ((long long)c << (cwsh - se[g])) + (kk >> se[g]) - 1;   // the group that closed
                        odst[nout + lv_] = m < sM[g] ? zs * a.R + soff[g] + (int)m : -1;
                    }
                    if (g) {
                        acc2 = f32x16{0};
                        acc3 = f32x16{0};
                    } else {
                        acc0 = f32x16{0};
                        acc1 = f32x16{0};
                    }
                }
                nout += cn;
            }
        }
        // The unit's output leaves in a few wide stores (a store retires in
        // order with the ring's loads, so every store instruction can hold up
        // the stream): its closed groups, 8 bf16 rows per store, ...
        FMA_FLUSH_ROWS();
        // ... and its fp32 part of every wider group, for coarsen_finish,
        // straight from the folded accumulators (16 bytes per lane and store)
#pragma unroll
        for (int g = 0; g < CG; ++g) {
            if (ndir >= nlev || 16 * g + 16 <= ndir || 16 * g >= nlev) continue;
            const int l = 16 * g + lv_;
            const bool wide = l >= ndir && l < nlev;
            float *const dst = a.part + (((long long)zs * a.npartial + ((wide ? l : ndir) - a.first_partial)) *
                                             a.part_count + c) * 64 + 32 * pt + 4 * h;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const f32x4 f = g ? fold_parts4(acc2, acc3, jj) : fold_parts4(acc0, acc1, jj);
                if (wide) *reinterpret_cast<f32x4 *>(dst + 8 * jj) = f;
            }
        }
        acc0 = f32x16{0};
        acc1 = f32x16{0};
        acc2 = f32x16{0};
        acc3 = f32x16{0};
    }
#undef FMA_FLUSH_ROWS
}

// 2D bf16 coarsening on the matrix cores (Eq. agg2d).  One wave per unit:
// a 32x32-pixel tile of one (tensor, slice), streamed row by row, 16 pixels
// (one contiguous 2 KB run) per step, through a ring of D slots filled by
// direct-to-LDS loads.  A slot holds the step's 16 pixel rows, the y weights
// of those 16 pixels for every set (16 per set, NWY loads of four sets each)
// and the x weight of the step's row for every set (one load).  Every
// accumulator column is one (set, square column of the tile): 32 / s of them
// for a set of square side s <= 32, one for a wider set.  Its B operand is
// wx[row] * wy[pixel] on the pixels of that square column and zero elsewhere,
// split into bf16 hi and lo columns as in the 1D kernel, so the columns hold
// each square's running sum in fp32.  Squares of side s <= 32 close after
// every s rows and are staged and written like the 1D groups; a wider square
// leaves the tile's fp32 part for coarsen_finish.
template <int D, int NWY, int CG>
__global__ __launch_bounds__(256) void coarsen2d_stream(CoarsenArgs a)
{
    extern __shared__ __attribute__((aligned(16))) unsigned char csm[];
    static_assert(D >= 2 && D <= 6 && NWY >= 1 && NWY <= 8 && (CG == 1 || CG == 2), "ring shape");
    constexpr int DATAB = 16 * 128;          // 16 bf16 pixel rows
    constexpr int WXB = DATAB + 256 * NWY;   // then the x weights of up to 64 sets
    constexpr int SLOTB = WXB + 256;
    constexpr int NLD = 3 + NWY;             // loads per step
    constexpr int NSTEP = 64;                // 32 rows x 2 halves
    const int nlev = a.lv.nlev;
    int ncols = 0, ndir = 0;                 // columns of the pass; sets of side <= 32 (a prefix)
    for (int e = 0; e < nlev; ++e) {
        ncols += stream2d_cols(a.lv.size[e]);
        if (a.lv.size[e] <= 32) ndir = e + 1;
    }
    // the host sizes each wave's LDS and picks the instance with the same
    // rules; a launch that does not match them does nothing
    if (a.wave_lds < stream2d_wave_lds(D, NWY) || nlev > 4 * NWY || ncols > 16 * CG) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // per wave: D slots | 64 zero bytes | 16 staged bf16 output rows | their
    // 16 row indices
    unsigned char *const ring = csm + wave * a.wave_lds;
    unsigned char *const zero = ring + D * SLOTB;
    __bf16 *const orow = reinterpret_cast<__bf16 *>(zero + 64);                  // [16][64]
    int *const odst = reinterpret_cast<int *>(zero + 64 + 2048);                 // [16]
    if (lane < 16) reinterpret_cast<float *>(zero)[lane] = 0.f;
    const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(
        static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void *)ring)));

    const int W = a.side, nty = a.tiles_y;             // tiles along y (columns); tile t = tx * nty + ty
    const int upz = a.nchunk;                          // tiles per (tensor, slice)
    const int U = 2 * a.nslice * upz;
    const int G = gridDim.x * 4;
    const int gw = blockIdx.x * 4 + wave;
    const long long rowstep = (long long)W * 128 - 2048;   // from the second half of a row to the next row

    // ---- issue side.  y-weight load i: lane L gathers pixel L % 16 of set
    // 4 i + L / 16; x-weight load: lane L gathers the row's weight of set L.
    // Lanes past the last set read weight 0 of the head.
    const uint32_t rowoff = (lane >> 3) * 128 + 16 * ((lane & 7) ^ (2 * ((lane >> 3) & 3)));
    const uint32_t rowoff8 = rowoff + 1024;   // pixels 8 .. 15 of the step
    int iu = gw, ist = 0, islot = 0;
    const char *isrc = nullptr;      // first pixel row of the step to issue (uniform)
    const float *ipi = nullptr;      // weight vectors of the unit's head (uniform)
    int iyo0[NWY], iyo1[NWY];        // y-weight offset of the lane's pixel in the first / second half
    int ixb = 0, ixm = 0;            // x-weight base and row mask of the lane's set
    // (the set table is read again at every unit start rather than kept in
    // registers through the stream)
#define FMA_UNIT_ISSUE_SETUP()                                                                          \
    do {                                                                                                \
        const int zs_ = iu / upz, t_ = iu - zs_ * upz;                                                  \
        const int z_ = zs_ >= a.nslice, sl_ = zs_ - z_ * a.nslice;                                      \
        const int tx_ = t_ / nty, ty_ = t_ - tx_ * nty;                                                 \
        isrc = static_cast<const char *>(z_ ? a.v : a.k) +                                              \
               ((long long)sl_ * a.n + (long long)(32 * tx_) * W + 32 * ty_) * 128;                     \
        ipi = (z_ ? a.wv : a.wk) + (long long)(sl_ % a.heads) * a.w_stride;                             \
        _Pragma("unroll") for (int i_ = 0; i_ < NWY; ++i_) {                                            \
            const int e_ = 4 * i_ + (lane >> 4), y_ = lane & 15;                                        \
            iyo0[i_] = 0;                                                                               \
            iyo1[i_] = 0;                                                                               \
            if (e_ < nlev) {                                                                            \
                const int s_ = a.lv.size[e_], b_ = a.lv.woff[e_] + s_;                                  \
                iyo0[i_] = s_ <= 32 ? b_ + (y_ & (s_ - 1)) : b_ + ((32 * ty_) & (s_ - 1)) + y_;         \
                iyo1[i_] = s_ <= 32 ? b_ + ((16 + y_) & (s_ - 1)) : b_ + ((32 * ty_) & (s_ - 1)) + 16 + y_; \
            }                                                                                           \
        }                                                                                               \
        ixb = 0;                                                                                        \
        ixm = 0;                                                                                        \
        if (lane < nlev) {                                                                              \
            const int s_ = a.lv.size[lane];                                                             \
            ixb = s_ <= 32 ? a.lv.woff[lane] : a.lv.woff[lane] + ((32 * tx_) & (s_ - 1));               \
            ixm = s_ <= 32 ? s_ - 1 : 31;                                                               \
        }                                                                                               \
    } while (0)
    if (iu < U) FMA_UNIT_ISSUE_SETUP();
    int issued = 0;   // steps issued, counted since the start
    auto issue_next = [&]() {
        if (iu >= U) return;
        const uint32_t dst = ring_lds + islot * SLOTB;
        const int hf = ist & 1, x = ist >> 1;
        dma16_sv(rowoff, isrc, dst);
        dma16_sv(rowoff8, isrc, dst + 1024);
#pragma unroll
        for (int i = 0; i < NWY; ++i) dma4_sv(4u * (uint32_t)(hf ? iyo1[i] : iyo0[i]), ipi, dst + DATAB + 256 * i);
        dma4_sv(4u * (uint32_t)(ixb + (x & ixm)), ipi, dst + WXB);
        ++issued;
        isrc += hf ? rowstep : 2048;
        islot = islot + 1 == D ? 0 : islot + 1;
        if (++ist == NSTEP) {
            ist = 0;
            iu += G;
            if (iu < U) FMA_UNIT_ISSUE_SETUP();
        }
    };
#undef FMA_UNIT_ISSUE_SETUP

    // ---- consume side: accumulator column c of group g is the lane's
    // (set, square column) number 16 g + c % 16, part c / 16
    const int col = lane & 31, lv_ = col & 15, pt = col >> 4, h = lane >> 5;
    int ce[CG], cj[CG];   // the lane's set (-1: none) and square column
#pragma unroll
    for (int g = 0; g < CG; ++g) {
        ce[g] = -1;
        cj[g] = 0;
    }
    {
        int c0 = 0;
        for (int e = 0; e < nlev; ++e) {
            const int nc = stream2d_cols(a.lv.size[e]);
#pragma unroll
            for (int g = 0; g < CG; ++g) {
                const int sc = 16 * g + lv_;
                if (sc >= c0 && sc < c0 + nc) {
                    ce[g] = e;
                    cj[g] = sc - c0;
                }
            }
            c0 += nc;
        }
    }
    // per group: the lane's weight offsets in a slot, which of its 8 k-slots
    // (pixels 4h .. 4h+3 and 8+4h .. 8+4h+3 of the step) lie in its square
    // column in each half, and its set's output geometry
    int wyr[CG], wxr[CG], mk0[CG], mk1[CG], sM[CG], sMy[CG], soff[CG], ssh[CG];
#pragma unroll
    for (int g = 0; g < CG; ++g) {
        const int e = ce[g];
        wyr[g] = e >= 0 ? DATAB + 64 * e + 16 * h : -1;
        wxr[g] = e >= 0 ? WXB + 4 * e : -1;
        sM[g] = 0;
        sMy[g] = 0;
        soff[g] = 0;
        ssh[g] = 0;
        int lo = 0, hi = 0;
        if (e >= 0) {
            const int sz = a.lv.size[e];
            sM[g] = a.lv.M[e];
            sMy[g] = a.lv.My[e];
            soff[g] = a.lv.off[e];
            ssh[g] = 31 - __builtin_clz(sz);
            lo = sz <= 32 ? cj[g] * sz : 0;
            hi = sz <= 32 ? lo + sz : 32;
        }
        int m0 = 0, m1 = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int y = i < 4 ? 4 * h + i : 8 + 4 * h + i - 4;
            m0 |= (y >= lo && y < hi) << i;
            m1 |= (16 + y >= lo && 16 + y < hi) << i;
        }
        mk0[g] = m0;
        mk1[g] = m1;
    }
    int voff[2];
    {
        const int gq = lane >> 4, s4 = lane & 15, j = s4 >> 2, q = s4 & 3;
        const int row = 4 * (gq >> 1) + j;
#pragma unroll
        for (int db = 0; db < 2; ++db) {
            const int ch = 4 * db + 2 * (gq & 1) + (q >> 1);
            voff[db] = row * 128 + 16 * (ch ^ (2 * (row & 3))) + 8 * (q & 1);
        }
    }

#pragma unroll
    for (int j = 0; j < D; ++j) issue_next();

    int consumed = 0, cslot = 0, nout = 0;
    // write the staged bf16 rows (8 per store instruction) and empty the staging
#define FMA_FLUSH_ROWS()                                                                                  \
    do {                                                                                                  \
        for (int k0 = 0; k0 < nout; k0 += 8) {                                                            \
            const int k = k0 + (lane >> 3);                                                               \
            const uint4 v = *reinterpret_cast<const uint4 *>(orow + k * 64 + 8 * (lane & 7));             \
            const int dk = odst[k];                                                                       \
            if (k < nout && dk >= 0)                                                                      \
                *reinterpret_cast<uint4 *>(static_cast<__bf16 *>(a.coarse) + (long long)dk * kHeadDim +     \
                                           8 * (lane & 7)) = v;                                           \
        }                                                                                                 \
        nout = 0;                                                                                         \
    } while (0)
    f32x16 acc[2 * CG];
#pragma unroll
    for (int i = 0; i < 2 * CG; ++i) acc[i] = f32x16{0};
    for (int cu = gw; cu < U; cu += G) {
        const int zs = cu / upz, t = cu - zs * upz;
        const int tx = t / nty, ty = t - tx * nty;
        for (int st = 0; st < NSTEP; ++st) {
            const int hf = st & 1, x = st >> 1;
            wait_oldest<NLD, D>(issued - consumed == D);
            const unsigned char *sl = ring + cslot * SLOTB;
            bf16x8 av[2];
#pragma unroll
            for (int db = 0; db < 2; ++db) {
                const s16x4c r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4c *)(sl + voff[db]));
                const s16x4c r2 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4c *)(sl + 8 * 128 + voff[db]));
                typedef short s16x8 __attribute__((ext_vector_type(8)));
                const s16x8 tt = {r1[0], r1[1], r1[2], r1[3], r2[0], r2[1], r2[2], r2[3]};
                av[db] = __builtin_bit_cast(bf16x8, tt);
            }
            f32x4 wy0[CG], wy1[CG];
            float wx[CG];
#pragma unroll
            for (int g = 0; g < CG; ++g) {
                const unsigned char *wp = wyr[g] >= 0 ? sl + wyr[g] : zero;
                wy0[g] = *reinterpret_cast<const f32x4 *>(wp);
                wy1[g] = *reinterpret_cast<const f32x4 *>(wp + 32);
                wx[g] = *reinterpret_cast<const float *>(wxr[g] >= 0 ? sl + wxr[g] : zero);
            }
            wait_lgkm0();   // the slot is read: refill it
            ++consumed;
            cslot = cslot + 1 == D ? 0 : cslot + 1;
            issue_next();
#pragma unroll
            for (int g = 0; g < CG; ++g) {
                const int m = hf ? mk1[g] : mk0[g];
                f32x4 w0, w1;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    w0[i] = (m >> i) & 1 ? wx[g] * wy0[g][i] : 0.f;
                    w1[i] = (m >> (4 + i)) & 1 ? wx[g] * wy1[g][i] : 0.f;
                }
                const bf16x8 bw = split_weights(w0, w1, pt);
                acc[2 * g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[0], bw, acc[2 * g], 0, 0, 0);
                acc[2 * g + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[1], bw, acc[2 * g + 1], 0, 0, 0);
            }
            if (!hf) continue;
            // squares that close with this row: those of a prefix of the sets
            // (the sides are ascending powers of two), i.e. a prefix of the
            // columns; folded and staged together, one column group at a time
            int lc = 0, lcc = 0;
            while (lc < ndir && !((x + 1) & (a.lv.size[lc] - 1))) {
                lcc += stream2d_cols(a.lv.size[lc]);
                ++lc;
            }
#pragma unroll
            for (int g = 0; g < CG; ++g) {
                const int cn = lcc - 16 * g < 16 ? lcc - 16 * g : 16;   // closing columns of this group
                if (cn <= 0) break;
                if (nout + cn > 16) FMA_FLUSH_ROWS();
                __bf16 *const dst = orow + (nout + (lv_ < cn ? lv_ : 0)) * 64 + 32 * pt + 4 * h;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const f32x4 f = fold_parts4(acc[2 * g], acc[2 * g + 1], jj);
                    if (lv_ < cn) *reinterpret_cast<uint2 *>(dst + 8 * jj) = uint2{cvt_pk_bf16(f[0], f[1]), cvt_pk_bf16(f[2], f[3])};
                }
                if (lv_ < cn) {
                    if (pt == 0 && h == 0) {
                        const int u = (32 * tx + x) >> ssh[g], v = ((32 * ty) >> ssh[g]) + cj[g];
                        odst[nout + lv_] = u < sM[g] && v < sMy[g] ? zs * a.R + soff[g] + u * sMy[g] + v : -1;
                    }
                    acc[2 * g] = f32x16{0};
                    acc[2 * g + 1] = f32x16{0};
                }
                nout += cn;
            }
        }
        FMA_FLUSH_ROWS();
        // the tile's fp32 part of every wider square, for coarsen_finish,
        // straight from the folded accumulators (16 bytes per lane and store)
        int dcols = 0;
        for (int e = 0; e < ndir; ++e) dcols += stream2d_cols(a.lv.size[e]);
#pragma unroll
        for (int g = 0; g < CG; ++g) {
            if (dcols >= ncols || 16 * g + 16 <= dcols || 16 * g >= ncols) continue;
            const bool wide = ce[g] >= ndir;
            float *const dst = a.part + (((long long)zs * a.npartial + ((wide ? ce[g] : ndir) - a.first_partial)) *
                                             a.part_count + t) * 64 + 32 * pt + 4 * h;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const f32x4 f = fold_parts4(acc[2 * g], acc[2 * g + 1], jj);
                if (wide) *reinterpret_cast<f32x4 *>(dst + 8 * jj) = f;
            }
        }
#pragma unroll
        for (int i = 0; i < 2 * CG; ++i) acc[i] = f32x16{0};
    }
#undef FMA_FLUSH_ROWS
}

// Sum the per-chunk partials of every group of the levels that span several
// chunks, in ascending chunk order.  One thread per (tensor, slice, group, channel).
template <bool BF16>
__global__ __launch_bounds__(256) void coarsen_finish(CoarsenArgs a, long long total, int rows_per_zs)
{
    const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
    if (idx >= total) return;
    const int D = a.head_dim;
    const int c = (int)(idx % D);
    const long long rowid = idx / D;
    const long long zs = rowid / rows_per_zs;
    int rem = (int)(rowid - zs * rows_per_zs);
    int l = a.first_partial;
    int groups = a.two_d ? a.lv.M[l] * a.lv.My[l] : a.lv.M[l];
    while (rem >= groups) {
        rem -= groups;
        ++l;
        groups = a.two_d ? a.lv.M[l] * a.lv.My[l] : a.lv.M[l];
    }
    const float *p = a.part + (zs * a.npartial + (l - a.first_partial)) * (long long)a.part_count * D + c;
    const int per = a.lv.size[l] / a.part_span;   // partials (2D: tiles along each axis) per group
    float sum = 0.f;
    if (!a.two_d) {
        const int m = rem;
        const int lo = m * per, hi = (m + 1) * per < a.part_count ? (m + 1) * per : a.part_count;
        // eight loads in flight; the sum is taken in ascending order
        int ch = lo;
        for (; ch + 8 <= hi; ch += 8) {
            float t[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) t[e] = p[(long long)(ch + e) * D];
#pragma unroll
            for (int e = 0; e < 8; ++e) sum += t[e];
        }
        for (; ch < hi; ++ch) sum += p[(long long)ch * D];
    } else {
        const int My = a.lv.My[l];
        const int u = rem / My, v = rem - u * My;
        for (int tx = u * per; tx < (u + 1) * per && tx < a.tiles_x; ++tx)
            for (int ty = v * per; ty < (v + 1) * per && ty < a.tiles_y; ++ty)
                sum += p[(long long)(tx * a.tiles_y + ty) * D];
    }
    store1<BF16>(a.coarse, (zs * a.R + a.lv.off[l] + rem) * D + c, sum);
}

// ---------------------------------------------------------------- 2D
// grid (tiles, nslice, 2).  A tile is 32x32 pixels cut into NRUN = NT / (D / 8)
// runs (D / 8 threads per pixel row, 8 channels each); thread `run` covers
// RX = (1024 / NRUN) / r pixel rows by RY = r columns of one base cell (the
// launcher takes NT >= 128 D / r^2, so that RX <= r and a run never
// straddles a square).
template <bool BF16, int NLEV, int NT, int D>
__global__ __launch_bounds__(NT) void coarsen2d_tiles(CoarsenArgs a)
{
    extern __shared__ __attribute__((aligned(16))) float smem[];
    constexpr int T = 32;
    constexpr int CPR = D / 8;
    constexpr int NRUN = NT / CPR;            // runs per tile
    const int tile = blockIdx.x, slice = blockIdx.y, z = blockIdx.z;
    const int tid = threadIdx.x, c8 = tid % CPR, run = tid / CPR;
    const int W = a.side, H = a.height, r = a.r;
    const int RY = r, RX = (T * T / NRUN) / r;   // run = RX x RY pixels
    const int rcols = T / RY;                  // runs per tile row band
    const int nty = a.tiles_y;
    const int tx = tile / nty, ty = tile - tx * nty;
    const int x0 = tx * T, y0 = ty * T;
    const float *pi = (z ? a.wv : a.wk) + (long long)(slice % a.heads) * a.w_stride;

    // weight windows along x and y: level l needs min(s_l, T) entries each
    int wxo[NLEV], wyo[NLEV], wlen[NLEV];
    int wtot = 0;
#pragma unroll
    for (int l = 0; l < NLEV; ++l) {
        const int s = a.lv.size[l];
        wlen[l] = s < T ? s : T;
        wxo[l] = wtot;
        wyo[l] = wtot + wlen[l];
        const int sx = s > T ? x0 % s : 0, sy = s > T ? y0 % s : 0;
        for (int t = tid; t < wlen[l]; t += NT) {
            smem[wxo[l] + t] = pi[a.lv.woff[l] + sx + t];
            smem[wyo[l] + t] = pi[a.lv.woff[l] + s + sy + t];
        }
        wtot += 2 * wlen[l];
    }
    float *red = smem + wtot;
    __syncthreads();

    const int rrow = run / rcols, rcol = run - rrow * rcols;
    const int xa = x0 + rrow * RX, ya = y0 + rcol * RY;
    const void *src = z ? a.v : a.k;
    const long long sbase = (long long)slice * a.n * D + c8 * 8;

    float acc[NLEV][8];
#pragma unroll
    for (int l = 0; l < NLEV; ++l)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[l][c] = 0.f;

    for (int dx = 0; dx < RX; ++dx) {
        const int x = xa + dx;
        if (x >= H) break;
        for (int dy = 0; dy < RY; dy += 4) {
            float xv[4][8];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int y = ya + dy + u;
                if (y < W) {
                    load8<BF16>(src, sbase + ((long long)x * W + y) * D, xv[u]);
                } else {
#pragma unroll
                    for (int c = 0; c < 8; ++c) xv[u][c] = 0.f;
                }
            }
#pragma unroll
            for (int l = 0; l < NLEV; ++l) {
                const float wx = smem[wxo[l] + (x - x0) % wlen[l]];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const float w = wx * smem[wyo[l] + (ya + dy + u - y0) % wlen[l]];
#pragma unroll
                    for (int c = 0; c < 8; ++c) acc[l][c] = fmaf(w, xv[u][c], acc[l][c]);
                }
            }
        }
    }

    const int zs = z * a.nslice + slice;
#pragma unroll
    for (int l = 0; l < NLEV; ++l) {
        float *buf = red + (l & 1) * NRUN * D;
        *reinterpret_cast<float4 *>(&buf[run * D + c8 * 8]) =
            make_float4(acc[l][0], acc[l][1], acc[l][2], acc[l][3]);
        *reinterpret_cast<float4 *>(&buf[run * D + c8 * 8 + 4]) =
            make_float4(acc[l][4], acc[l][5], acc[l][6], acc[l][7]);
        __syncthreads();
        const int s = a.lv.size[l];
        if (s <= T) {
            const int G = T / s;                         // squares per tile side
            const int rpx = s / RX, rpy = s / RY;        // runs per square along x, y
            for (int o = tid; o < G * G * D; o += NT) {
                const int sq = o / D, c = o - sq * D;
                const int su = sq / G, sv = sq - su * G;
                float sum = 0.f;
                for (int i = 0; i < rpx; ++i)
                    for (int j = 0; j < rpy; ++j)
                        sum += buf[((su * rpx + i) * rcols + (sv * rpy + j)) * D + c];
                const int M = a.lv.M[l], My = a.lv.My[l];
                const int u = tx * G + su, v = ty * G + sv;
                if (u < M && v < My)
                    store1<BF16>(a.coarse, ((long long)zs * a.R + a.lv.off[l] + u * My + v) * D + c, sum);
            }
        } else if (tid < D) {
            float sum = 0.f;
            for (int t = 0; t < NRUN; ++t) sum += buf[t * D + tid];
            const long long pl = l - a.first_partial;
            a.part[(((long long)zs * a.npartial + pl) * a.part_count + tile) * D + tid] = sum;
        }
    }
}

// ---------------------------------------------------------------- launchers
// The streaming kernel's grid: as many waves as fit on the device (occupancy
// of the kernel at its LDS size, cached per device by resident_slots), then trimmed so that
// every wave gets the same number of units, up to one.
template <int D, int NWD>
static hipError_t launch_stream_dn(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    const int slots = resident_slots(reinterpret_cast<const void *>(&coarsen1d_stream<D, NWD>), 256, smem);
    if (slots <= 0) return hipErrorInvalidDevice;
    const long long units = 2LL * a.nslice * a.nchunk;
    const long long cap = 4LL * slots;
    const long long per_wave = (units + cap - 1) / cap;
    const long long waves = (units + per_wave - 1) / per_wave;
    const unsigned grid = (unsigned)((waves + 3) / 4);
    hipLaunchKernelGGL((coarsen1d_stream<D, NWD>), dim3(grid), dim3(256), smem, st, a);
    return hipGetLastError();
}

template <int NWD>
static hipError_t launch_stream_n(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    switch (a.depth) {
    case 2: return launch_stream_dn<2, NWD>(a, st, smem);
    case 3: return launch_stream_dn<3, NWD>(a, st, smem);
    case 4: return launch_stream_dn<4, NWD>(a, st, smem);
    case 5: return launch_stream_dn<5, NWD>(a, st, smem);
    case 6: return launch_stream_dn<6, NWD>(a, st, smem);
    default: return hipErrorInvalidValue;
    }
}

static hipError_t launch_stream(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    switch (stream_weight_loads(a.lv.nlev)) {
    case 1: return launch_stream_n<1>(a, st, smem);
    case 2: return launch_stream_n<2>(a, st, smem);
    case 3: return launch_stream_n<3>(a, st, smem);
    case 4: return launch_stream_n<4>(a, st, smem);
    case 6: return launch_stream_n<6>(a, st, smem);
    case 8: return launch_stream_n<8>(a, st, smem);
    default: return hipErrorInvalidValue;
    }
}

template <int D, int NWY, int CG>
static hipError_t launch_stream2d_d(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    const int slots = resident_slots(reinterpret_cast<const void *>(&coarsen2d_stream<D, NWY, CG>), 256, smem);
    if (slots <= 0) return hipErrorInvalidDevice;
    const long long units = 2LL * a.nslice * a.nchunk;
    const long long cap = 4LL * slots;
    const long long per_wave = (units + cap - 1) / cap;
    const long long waves = (units + per_wave - 1) / per_wave;
    const unsigned grid = (unsigned)((waves + 3) / 4);
    hipLaunchKernelGGL((coarsen2d_stream<D, NWY, CG>), dim3(grid), dim3(256), smem, st, a);
    return hipGetLastError();
}

template <int NWY, int CG>
static hipError_t launch_stream2d_n(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    switch (a.depth) {
    case 2: return launch_stream2d_d<2, NWY, CG>(a, st, smem);
    case 3: return launch_stream2d_d<3, NWY, CG>(a, st, smem);
    case 4: return launch_stream2d_d<4, NWY, CG>(a, st, smem);
    default: return hipErrorInvalidValue;
    }
}

template <int CG>
static hipError_t launch_stream2d_c(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    switch (stream2d_weight_loads(a.lv.nlev)) {
    case 1: return launch_stream2d_n<1, CG>(a, st, smem);
    case 2: return launch_stream2d_n<2, CG>(a, st, smem);
    case 4: return launch_stream2d_n<4, CG>(a, st, smem);
    case 8: return launch_stream2d_n<8, CG>(a, st, smem);
    default: return hipErrorInvalidValue;
    }
}

static hipError_t launch_stream2d(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    int cols = 0;
    for (int e = 0; e < a.lv.nlev; ++e) cols += stream2d_cols(a.lv.size[e]);
    if (cols <= 16) return launch_stream2d_c<1>(a, st, smem);
    if (cols <= 32) return launch_stream2d_c<2>(a, st, smem);
    return hipErrorInvalidValue;
}

template <bool BF16, int NLEV, int D>
static hipError_t launch_coarsen_nd(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    const dim3 grid(a.nchunk, a.nslice, 2);
    // workgroup size by cell side and head dim (coarsen2d_threads): 4 x 4
    // cells take 512 threads at d = 64 and 1024 at d = 128, all else 256
    constexpr int NT4 = D == 128 ? 1024 : D == 64 ? 512 : 256;
    static_assert(NT4 == coarsen2d_threads(4, D) && coarsen2d_threads(8, D) == 256, "tile threads");
    if (!a.two_d)
        hipLaunchKernelGGL((coarsen1d_chunks<BF16, NLEV, D>), grid, dim3(256), smem, st, a);
    else if (a.r < 8)
        hipLaunchKernelGGL((coarsen2d_tiles<BF16, NLEV, NT4, D>), grid, dim3(NT4), smem, st, a);
    else
        hipLaunchKernelGGL((coarsen2d_tiles<BF16, NLEV, 256, D>), grid, dim3(256), smem, st, a);
    return hipGetLastError();
}

template <bool BF16, int NLEV>
static hipError_t launch_coarsen_n(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    switch (a.head_dim) {
    case 32: return launch_coarsen_nd<BF16, NLEV, 32>(a, st, smem);
    case 64: return launch_coarsen_nd<BF16, NLEV, 64>(a, st, smem);
    case 128: return launch_coarsen_nd<BF16, NLEV, 128>(a, st, smem);
    default: return hipErrorInvalidValue;
    }
}

template <bool BF16>
static hipError_t launch_coarsen_t(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    switch (a.lv.nlev) {
#define FMA_CASE(N) case N: return launch_coarsen_n<BF16, N>(a, st, smem);
        FMA_CASE(1) FMA_CASE(2) FMA_CASE(3) FMA_CASE(4) FMA_CASE(5) FMA_CASE(6)
        FMA_CASE(7) FMA_CASE(8) FMA_CASE(9) FMA_CASE(10) FMA_CASE(11) FMA_CASE(12)
        FMA_CASE(13) FMA_CASE(14) FMA_CASE(15) FMA_CASE(16)
#undef FMA_CASE
    default: return hipErrorInvalidValue;
    }
}

// Coarse sets are built in passes of consecutive sets, each pass reading K
// and V once: at most kStreamSets per pass on the 1D bf16 streaming kernel
// (one pass whenever rank * (L - 1) <= 32), as many as fill 32 accumulator
// columns on the 2D one, kPassSets on the others.  A pass sees its sets as a
// table of its own; its partial sums keep their global index (first_partial
// is shifted by the pass's first set).
hipError_t launch_coarsen(const CoarsenArgs &a, bool bf16, size_t smem_bytes, hipStream_t st)
{
    if (a.nslice == 0 || a.nchunk == 0 || a.lv.nlev == 0) return hipSuccess;
    const bool stream = bf16 && a.depth > 0;
    hipError_t e = hipSuccess;
    for (int v0 = 0; v0 < a.lv.nlev && e == hipSuccess;) {
        int cnt = a.lv.nlev - v0;
        if (stream && a.two_d) {
            int cols = 0;
            cnt = 0;
            while (v0 + cnt < a.lv.nlev && cols + stream2d_cols(a.lv.size[v0 + cnt]) <= 32)
                cols += stream2d_cols(a.lv.size[v0 + cnt++]);
        } else {
            const int pass = stream ? kStreamSets : kPassSets;
            cnt = cnt < pass ? cnt : pass;
        }
        if (cnt <= 0) return hipErrorInvalidValue;
        CoarsenArgs b = a;
        memset(&b.lv, 0, sizeof(b.lv));
        b.lv.nlev = cnt;
        for (int i = 0; i < cnt; ++i) {
            b.lv.off[i] = a.lv.off[v0 + i];
            b.lv.M[i] = a.lv.M[v0 + i];
            b.lv.My[i] = a.lv.My[v0 + i];
            b.lv.size[i] = a.lv.size[v0 + i];
            b.lv.woff[i] = a.lv.woff[v0 + i];
            b.lv.lvl[i] = a.lv.lvl[v0 + i];
        }
        b.first_partial = a.first_partial - v0;
        if (stream)
            e = a.two_d ? launch_stream2d(b, st, smem_bytes) : launch_stream(b, st, smem_bytes);
        else
            e = bf16 ? launch_coarsen_t<true>(b, st, smem_bytes) : launch_coarsen_t<false>(b, st, smem_bytes);
        v0 += cnt;
    }
    if (e != hipSuccess) return e;
    if (a.first_partial < a.lv.nlev) {
        int rows = 0;
        for (int l = a.first_partial; l < a.lv.nlev; ++l)
            rows += a.two_d ? a.lv.M[l] * a.lv.My[l] : a.lv.M[l];
        const long long total = 2LL * a.nslice * rows * a.head_dim;
        const unsigned blocks = (unsigned)((total + 255) / 256);
        if (bf16)
            hipLaunchKernelGGL((coarsen_finish<true>), dim3(blocks), dim3(256), 0, st, a, total, rows);
        else
            hipLaunchKernelGGL((coarsen_finish<false>), dim3(blocks), dim3(256), 0, st, a, total, rows);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace fma_dev
