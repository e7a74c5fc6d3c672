// coarsen.hip -- per-level coarse keys/values (Eq. agg1d, Eq. agg2d) on gfx950.
//
// Every level is built straight from the fine tokens, so K and V are read
// from HBM exactly once.  A workgroup owns a chunk of CH consecutive tokens
// (1D) or a 32x32 tile of the token map (2D) of one (batch, head, tensor).
// Each thread streams a "run" of rows for 8 channels (16-byte loads, eight
// threads cover one 128-byte row) and keeps one fp32 partial sum per level
// and channel in registers; a run never crosses a base block, so it lies in
// exactly one group of every level.  The runs of a group are then summed in
// LDS in a fixed order.  Levels whose groups are larger than the chunk write
// one fp32 partial per chunk, and a second small kernel adds the partials of
// each group in ascending chunk order: no atomics, bitwise reproducible.
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
// grid (nchunk, nslice, 2): blockIdx.z selects K (0) or V (1).
template <bool BF16, int NLEV>
__global__ __launch_bounds__(256) void coarsen1d_chunks(CoarsenArgs a)
{
    extern __shared__ __attribute__((aligned(16))) float smem[];
    const int chunk = blockIdx.x, slice = blockIdx.y, z = blockIdx.z;
    const int tid = threadIdx.x, c8 = tid & 7, run = tid >> 3;
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
    float *red = smem + wtot;   // [2][32 runs][64 channels]
    __syncthreads();

    const long long row0 = (long long)chunk * CH + (long long)run * RUN;
    const void *src = z ? a.v : a.k;
    const long long sbase = (long long)slice * n * kHeadDim + c8 * 8;

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
        cur[u] = row < n ? load_raw<BF16>(src, sbase + row * kHeadDim) : zero_raw<BF16>();
    }
    for (int rr = 0; rr < RUN; rr += 4) {
        if (rr + 4 < RUN) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const long long row = row0 + rr + 4 + u;
                nxt[u] = row < n ? load_raw<BF16>(src, sbase + row * kHeadDim) : zero_raw<BF16>();
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
        float *buf = red + (l & 1) * 32 * 64;
        *reinterpret_cast<float4 *>(&buf[run * 64 + c8 * 8]) =
            make_float4(acc[l][0], acc[l][1], acc[l][2], acc[l][3]);
        *reinterpret_cast<float4 *>(&buf[run * 64 + c8 * 8 + 4]) =
            make_float4(acc[l][4], acc[l][5], acc[l][6], acc[l][7]);
        __syncthreads();
        const int s = a.lv.size[l];
        if (s <= CH) {
            const int G = CH / s, rpg = s / RUN;
            for (int o = tid; o < G * 64; o += 256) {
                const int g = o >> 6, c = o & 63;
                float sum = 0.f;
                for (int t = 0; t < rpg; ++t) sum += buf[(g * rpg + t) * 64 + c];
                const long long m = (long long)chunk * G + g;
                if (m < a.lv.M[l])
                    store1<BF16>(kbar, ((long long)zs * a.R + a.lv.off[l] + m) * kHeadDim + c, sum);
            }
        } else if (tid < 64) {
            float sum = 0.f;
            for (int t = 0; t < 32; ++t) sum += buf[t * 64 + tid];
            const long long pl = l - a.first_partial;
            a.part[(((long long)zs * a.npartial + pl) * a.part_count + chunk) * 64 + tid] = sum;
        }
    }
}

// bf16 1D coarsening with a per-wave prefetch ring in LDS.  The thread and
// run layout is that of coarsen1d_chunks, but rows travel HBM -> LDS with
// 16-byte direct-to-LDS loads issued D rows ahead: at step i the wave's
// eight runs need row i of each run, which is exactly one load of eight
// 128-byte rows, and every lane reads back the 16 bytes it fetched itself.
// No barrier in the streaming loop and no registers spent on the loads in
// flight.
__device__ inline void dma16_row(const void *gptr, uint32_t lds_base)
{
    asm volatile("global_load_lds_dwordx4 %0, off" : : "v"(gptr), "{m0}"(lds_base) : "memory");
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

template <int NLEV, int D>
__global__ __launch_bounds__(256) void coarsen1d_ring(CoarsenArgs a)
{
    extern __shared__ __attribute__((aligned(16))) float smem[];
    const int chunk = blockIdx.x, slice = blockIdx.y, z = blockIdx.z;
    const int tid = threadIdx.x, c8 = tid & 7, run = tid >> 3, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
        wtot += wlen[l];
    }
    // LDS: weight windows, then one ring of D rows per wave; after the
    // stream the rings hold the [2][32 runs][64 channels] reduction buffer
    const int ring_off = (wtot + 3) & ~3;
    unsigned char *ring = reinterpret_cast<unsigned char *>(smem + ring_off) + wave * D * 1024;
    float *red = smem + ring_off;

    // runs lie inside base blocks, so a run is either entirely in the
    // sequence or entirely past its end (then it streams row 0 and adds 0)
    const long long row0 = (long long)chunk * CH + (long long)run * RUN;
    const bool valid = row0 < n;
    const char *src = static_cast<const char *>(z ? a.v : a.k) +
                      ((long long)slice * n + (valid ? row0 : 0)) * (kHeadDim * 2) + c8 * 16;
    const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(
        static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void *)ring)));

#pragma unroll
    for (int l = 0; l < NLEV; ++l) {
        const int s = a.lv.size[l];
        const long long start = s > CH ? ((long long)chunk * CH) % s : 0;
        for (int t = tid; t < wlen[l]; t += 256) smem[wlo[l] + t] = pi[a.lv.woff[l] + start + t];
    }

    int wb[NLEV];
#pragma unroll
    for (int l = 0; l < NLEV; ++l) wb[l] = wlo[l] + (run * RUN) % wlen[l];
    float acc[NLEV][8];
#pragma unroll
    for (int l = 0; l < NLEV; ++l)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[l][c] = 0.f;

    __syncthreads();   // weight windows in LDS
#pragma unroll
    for (int j = 0; j < D; ++j)
        if (j < RUN) dma16_row(src + (long long)j * (kHeadDim * 2), ring_lds + j * 1024);

    for (int j = 0; j < RUN; j += 4) {
        float w[NLEV][4];
#pragma unroll
        for (int l = 0; l < NLEV; ++l) {
            // weights of rows j .. j+3 (16-byte aligned: window bases and run
            // offsets are multiples of 4 floats)
            const float4 w4 = *reinterpret_cast<const float4 *>(&smem[wb[l] + j]);
            w[l][0] = w4.x;
            w[l][1] = w4.y;
            w[l][2] = w4.z;
            w[l][3] = w4.w;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = j + u;
            // refill the slot consumed in the previous step (its read is done)
            if (i >= 1 && i - 1 + D < RUN) {
                wait_lgkm0();
                dma16_row(src + (long long)(i - 1 + D) * (kHeadDim * 2), ring_lds + ((i - 1) % D) * 1024);
            }
            // row i has landed when at most the rows issued after it are in flight
            if (i + D <= RUN)
                wait_vm<D - 1>();
            else
                wait_vm<0>();
            const uint4 raw = *reinterpret_cast<const uint4 *>(ring + (i % D) * 1024 + lane * 16);
            float x[8];
            x[0] = bf16lo_to_f32(raw.x); x[1] = bf16hi_to_f32(raw.x);
            x[2] = bf16lo_to_f32(raw.y); x[3] = bf16hi_to_f32(raw.y);
            x[4] = bf16lo_to_f32(raw.z); x[5] = bf16hi_to_f32(raw.z);
            x[6] = bf16lo_to_f32(raw.w); x[7] = bf16hi_to_f32(raw.w);
#pragma unroll
            for (int l = 0; l < NLEV; ++l)
#pragma unroll
                for (int c = 0; c < 8; ++c) acc[l][c] = fmaf(w[l][u], x[c], acc[l][c]);
        }
    }
    if (!valid) {
#pragma unroll
        for (int l = 0; l < NLEV; ++l)
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[l][c] = 0.f;
    }

    __syncthreads();   // every wave is done with its ring

    // Per level, the 32 runs' sums go to LDS; each group of runs is then
    // summed in ascending order and stored, or, for groups wider than the
    // chunk, left as the chunk's fp32 partial for the finish kernel.
    const int zs = z * a.nslice + slice;
#pragma unroll
    for (int l = 0; l < NLEV; ++l) {
        float *buf = red + (l & 1) * 32 * 64;
        *reinterpret_cast<float4 *>(&buf[run * 64 + c8 * 8]) =
            make_float4(acc[l][0], acc[l][1], acc[l][2], acc[l][3]);
        *reinterpret_cast<float4 *>(&buf[run * 64 + c8 * 8 + 4]) =
            make_float4(acc[l][4], acc[l][5], acc[l][6], acc[l][7]);
        __syncthreads();
        const int s = a.lv.size[l];
        if (s <= CH) {
            const int G = CH / s, rpg = s / RUN;
            for (int o = tid; o < G * 64; o += 256) {
                const int g = o >> 6, c = o & 63;
                float sum = 0.f;
                for (int t = 0; t < rpg; ++t) sum += buf[(g * rpg + t) * 64 + c];
                const long long m = (long long)chunk * G + g;
                if (m < a.lv.M[l])
                    store1<true>(a.coarse, ((long long)zs * a.R + a.lv.off[l] + m) * kHeadDim + c, sum);
            }
        } else if (tid < 64) {
            float sum = 0.f;
            for (int t = 0; t < 32; ++t) sum += buf[t * 64 + tid];
            const long long pl = l - a.first_partial;
            a.part[(((long long)zs * a.npartial + pl) * a.part_count + chunk) * 64 + tid] = sum;
        }
    }
}

// Sum the per-chunk partials of every group of the levels that span several
// chunks, in ascending chunk order.  One thread per (tensor, slice, group, channel).
template <bool BF16>
__global__ __launch_bounds__(256) void coarsen_finish(CoarsenArgs a, long long total, int rows_per_zs)
{
    const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
    if (idx >= total) return;
    const int c = (int)(idx & 63);
    const long long rowid = idx >> 6;
    const long long zs = rowid / rows_per_zs;
    int rem = (int)(rowid - zs * rows_per_zs);
    int l = a.first_partial;
    int groups = a.two_d ? a.lv.M[l] * a.lv.M[l] : a.lv.M[l];
    while (rem >= groups) {
        rem -= groups;
        ++l;
        groups = a.two_d ? a.lv.M[l] * a.lv.M[l] : a.lv.M[l];
    }
    const float *p = a.part + (zs * a.npartial + (l - a.first_partial)) * (long long)a.part_count * 64 + c;
    const int per = a.lv.size[l] / a.part_span;   // partials (2D: tiles per side) per group
    float sum = 0.f;
    if (!a.two_d) {
        const int m = rem;
        const int lo = m * per, hi = (m + 1) * per < a.part_count ? (m + 1) * per : a.part_count;
        // eight loads in flight; the sum is taken in ascending order
        int ch = lo;
        for (; ch + 8 <= hi; ch += 8) {
            float t[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) t[e] = p[(long long)(ch + e) * 64];
#pragma unroll
            for (int e = 0; e < 8; ++e) sum += t[e];
        }
        for (; ch < hi; ++ch) sum += p[(long long)ch * 64];
    } else {
        const int M = a.lv.M[l];
        const int u = rem / M, v = rem - u * M;
        const int nt = a.tiles_per_side;
        for (int tx = u * per; tx < (u + 1) * per && tx < nt; ++tx)
            for (int ty = v * per; ty < (v + 1) * per && ty < nt; ++ty)
                sum += p[(long long)(tx * nt + ty) * 64];
    }
    store1<BF16>(a.coarse, (zs * a.R + a.lv.off[l] + rem) * kHeadDim + c, sum);
}

// ---------------------------------------------------------------- 2D
// grid (tiles, nslice, 2).  A tile is 32x32 pixels; thread `run` covers
// RX = 32/r pixel rows by RY = r columns of one base cell.
template <bool BF16, int NLEV>
__global__ __launch_bounds__(256) void coarsen2d_tiles(CoarsenArgs a)
{
    extern __shared__ __attribute__((aligned(16))) float smem[];
    constexpr int T = 32;
    const int tile = blockIdx.x, slice = blockIdx.y, z = blockIdx.z;
    const int tid = threadIdx.x, c8 = tid & 7, run = tid >> 3;
    const int W = a.side, r = a.r;
    const int RY = r, RX = 32 / r;            // run = RX x RY pixels, RX * RY = 32
    const int rcols = T / RY;                  // runs per tile row band
    const int nt = a.tiles_per_side;
    const int tx = tile / nt, ty = tile - tx * nt;
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
        for (int t = tid; t < wlen[l]; t += 256) {
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
    const long long sbase = (long long)slice * a.n * kHeadDim + c8 * 8;

    float acc[NLEV][8];
#pragma unroll
    for (int l = 0; l < NLEV; ++l)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[l][c] = 0.f;

    for (int dx = 0; dx < RX; ++dx) {
        const int x = xa + dx;
        if (x >= W) break;
        for (int dy = 0; dy < RY; dy += 4) {
            float xv[4][8];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int y = ya + dy + u;
                if (y < W) {
                    load8<BF16>(src, sbase + ((long long)x * W + y) * kHeadDim, xv[u]);
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
        float *buf = red + (l & 1) * 32 * 64;
        *reinterpret_cast<float4 *>(&buf[run * 64 + c8 * 8]) =
            make_float4(acc[l][0], acc[l][1], acc[l][2], acc[l][3]);
        *reinterpret_cast<float4 *>(&buf[run * 64 + c8 * 8 + 4]) =
            make_float4(acc[l][4], acc[l][5], acc[l][6], acc[l][7]);
        __syncthreads();
        const int s = a.lv.size[l];
        if (s <= T) {
            const int G = T / s;                         // squares per tile side
            const int rpx = s / RX, rpy = s / RY;        // runs per square along x, y
            for (int o = tid; o < G * G * 64; o += 256) {
                const int sq = o >> 6, c = o & 63;
                const int su = sq / G, sv = sq - su * G;
                float sum = 0.f;
                for (int i = 0; i < rpx; ++i)
                    for (int j = 0; j < rpy; ++j)
                        sum += buf[((su * rpx + i) * rcols + (sv * rpy + j)) * 64 + c];
                const int M = a.lv.M[l];
                const int u = tx * G + su, v = ty * G + sv;
                if (u < M && v < M)
                    store1<BF16>(a.coarse, ((long long)zs * a.R + a.lv.off[l] + u * M + v) * kHeadDim + c, sum);
            }
        } else if (tid < 64) {
            float sum = 0.f;
            for (int t = 0; t < 32; ++t) sum += buf[t * 64 + tid];
            const long long pl = l - a.first_partial;
            a.part[(((long long)zs * a.npartial + pl) * a.part_count + tile) * 64 + tid] = sum;
        }
    }
}

// ---------------------------------------------------------------- launchers
template <bool BF16, int NLEV>
static hipError_t launch_coarsen_n(const CoarsenArgs &a, hipStream_t st, size_t smem)
{
    const dim3 grid(a.nchunk, a.nslice, 2);
    if (a.two_d)
        hipLaunchKernelGGL((coarsen2d_tiles<BF16, NLEV>), grid, dim3(256), smem, st, a);
    else if (BF16 && a.ring == 8)
        hipLaunchKernelGGL((coarsen1d_ring<NLEV, 8>), grid, dim3(256), smem, st, a);
    else if (BF16 && a.ring == 4)
        hipLaunchKernelGGL((coarsen1d_ring<NLEV, 4>), grid, dim3(256), smem, st, a);
    else
        hipLaunchKernelGGL((coarsen1d_chunks<BF16, NLEV>), grid, dim3(256), smem, st, a);
    return hipGetLastError();
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

hipError_t launch_coarsen(const CoarsenArgs &a, bool bf16, size_t smem_bytes, hipStream_t st)
{
    if (a.nslice == 0 || a.nchunk == 0 || a.lv.nlev == 0) return hipSuccess;
    hipError_t e = bf16 ? launch_coarsen_t<true>(a, st, smem_bytes)
                        : launch_coarsen_t<false>(a, st, smem_bytes);
    if (e != hipSuccess) return e;
    if (a.first_partial < a.lv.nlev) {
        int rows = 0;
        for (int l = a.first_partial; l < a.lv.nlev; ++l)
            rows += a.two_d ? a.lv.M[l] * a.lv.M[l] : a.lv.M[l];
        const long long total = 2LL * a.nslice * rows * 64;
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
