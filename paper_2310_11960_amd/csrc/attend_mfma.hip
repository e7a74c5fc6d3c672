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
#include "fma_device.hpp"
#include "fma_kernels.hpp"

namespace fma_dev {

namespace {

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void gbl_void;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int KT = 64;             // keys per tile
constexpr int ROWB = 128;          // bytes of one bf16 row (64 channels)
constexpr int TILEB = KT * ROWB;   // one K or V tile, 8 KB
constexpr int NSTAGE = 2;          // LDS buffers per tensor
constexpr int MAX_CTILES = 7;      // coarse tiles: ceil(27 * 16 / 64)
constexpr int MAX_SLOTS = MAX_CTILES * KT;

struct Smem {
    unsigned char k[NSTAGE][TILEB];
    unsigned char v[NSTAGE][TILEB];
    int crow[MAX_SLOTS];                    // coarse slot -> coarse row, -1 if empty
    unsigned long long cmask[MAX_CTILES];   // validity bit per slot of each coarse tile
};

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

// Workgroup id -> logical tile id.  Hardware hands out consecutive
// workgroup ids round-robin over the 8 XCDs; this bijection gives each XCD
// one contiguous range of tiles, so neighbouring query tiles (which read
// the same near-field K/V) share an L2.
__device__ inline int xcd_remap(int wg, int total)
{
    const int q = total >> 3, rem = total & 7;
    const int x = wg & 7, k = wg >> 3;
    return x < rem ? x * (q + 1) + k : rem * (q + 1) + (x - rem) * q + k;
}

template <int NW, int GEOM>
__global__ __launch_bounds__(64 * NW) void attend_mfma_kernel(AttnArgs a)
{
    constexpr int NT = 64 * NW;
    __shared__ Smem sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int hh = lane >> 5, l32 = lane & 31;

    const int wg = xcd_remap(blockIdx.x, gridDim.x);
    const int slice = wg / a.tiles_per_slice;
    const int qt = wg - slice * a.tiles_per_slice;

    const char *kg = static_cast<const char *>(a.k) + (long long)slice * a.n * ROWB;
    const char *vg = static_cast<const char *>(a.v) + (long long)slice * a.n * ROWB;

    // ------------------------------------------------ tile list of this query tile
    int nnear;                 // near-field tiles
    long long klo = 0;         // 1D / dense: first near key
    int cx = 0, cy = 0;        // 2D: query cell
    int dx0 = 0, dy0 = 0, ncy = 1, tpc = 1, lg_r = 0;   // 2D near-cell enumeration
    if constexpr (GEOM == GEOM_2D) {
        cx = qt / a.nbx;
        cy = qt - cx * a.nbx;
        dx0 = cx > 0 ? -1 : 0;
        const int dx1 = cx + 1 < a.nbx ? 1 : 0;
        dy0 = cy > 0 ? -1 : 0;
        const int dy1 = cy + 1 < a.nbx ? 1 : 0;
        ncy = dy1 - dy0 + 1;
        tpc = (a.r * a.r) / KT;
        lg_r = 31 - __builtin_clz(a.r);
        nnear = (dx1 - dx0 + 1) * ncy * tpc;
    } else if constexpr (GEOM == GEOM_1D) {
        klo = qt > 0 ? (long long)(qt - 1) * a.r : 0;
        long long hi = a.causal ? (long long)(qt + 1) * a.r : (long long)(qt + 2) * a.r;
        if (hi > a.n) hi = a.n;
        nnear = (int)((hi - klo) / KT);
    } else {
        long long hi = a.causal ? (long long)(qt + 1) * a.qtile : a.n;
        if (hi > a.n) hi = a.n;
        nnear = (int)((hi + KT - 1) / KT);
    }
    const int nslot = a.nslot;
    const int nctile = (nslot + KT - 1) / KT;
    const int ntiles = nnear + nctile;

    // ------------------------------------------------ coarse slot table
    // slot lev * K + j holds list entry j of level lev + 1; levels are walked
    // in a uniform loop so the per-level tables are read with scalar loads.
    if (nctile > 0) {
        constexpr int K = GEOM == GEOM_2D ? kSlots2D : kSlots1D;
        for (int t = tid; t < nctile * KT; t += NT) sm.crow[t] = -1;
        __syncthreads();
        const int nlev = a.lv.nlev;
        for (int lev = 0; lev < nlev; ++lev) {
            const int M = a.lv.M[lev], off = a.lv.off[lev];
            if (tid < K) {
                int g;
                if constexpr (GEOM == GEOM_2D)
                    g = list2d_entry(cx, cy, lev + 1, tid, M);
                else
                    g = list1d_entry(qt, lev + 1, tid, M, a.causal);
                if (g >= 0) sm.crow[lev * K + tid] = off + g;
            }
        }
        __syncthreads();
        for (int ct = wave; ct < nctile; ct += NW) {
            const unsigned long long m = __builtin_amdgcn_ballot_w64(sm.crow[ct * KT + lane] >= 0);
            if (lane == 0) sm.cmask[ct] = m;
        }
    }
    const char *kbar = static_cast<const char *>(a.kbar) + (long long)slice * a.R * ROWB;
    const char *vbar = static_cast<const char *>(a.vbar) + (long long)slice * a.R * ROWB;

    // ------------------------------------------------ this lane's query (B operand Q^T)
    const int ql = wave * 32 + l32;
    long long qtok;
    if constexpr (GEOM == GEOM_2D) {
        const int pa = ql >> lg_r, pb = ql & (a.r - 1);
        qtok = (long long)(cx * a.r + pa) * a.side + (cy * a.r + pb);
    } else {
        qtok = (long long)qt * a.qtile + ql;
    }
    const long long qrow = ((long long)slice * a.n + qtok) * kHeadDim;
    bf16x8 qb[4];
    {
        const __bf16 *qp = static_cast<const __bf16 *>(a.q) + qrow;
#pragma unroll
        for (int c = 0; c < 4; ++c) qb[c] = *reinterpret_cast<const bf16x8 *>(qp + 16 * c + 8 * hh);
    }
    const long long wave_q0 = (long long)qt * a.qtile + wave * 32;   // 1D: first query of this wave

    // ------------------------------------------------ per-lane LDS offsets
    // direct loads: lane writes chunk position (lane & 7) of tile row 8i + (lane >> 3)
    const int lrow = lane >> 3;
    const int ldk0 = lrow * ROWB + 16 * ((lane & 7) ^ lrow);            // i even
    const int ldk1 = lrow * ROWB + 16 * ((lane & 7) ^ lrow ^ 1);        // i odd
    const int ldv = lrow * ROWB + 16 * ((lane & 7) ^ (2 * (lrow & 3)));
    // K operand reads: row l32 of a 32-key block, logical chunk 2*c4 + hh
    int koff[4];
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) koff[c4] = l32 * ROWB + 16 * ((2 * c4 + hh) ^ swz_k(l32));
    // V^T operand reads (transposing load): see the header comment
    int voff[2];
    {
        const int g = lane >> 4, s = lane & 15, j = s >> 2, q = s & 3;
        const int row = 4 * (g >> 1) + j;
#pragma unroll
        for (int db = 0; db < 2; ++db) {
            const int chunk = 4 * db + 2 * (g & 1) + (q >> 1);
            voff[db] = row * ROWB + 16 * (chunk ^ swz_v(row)) + 8 * (q & 1);
        }
    }

    // ------------------------------------------------ tile loads (direct to LDS)
    // Tile t: instructions 0..7 load K rows 8i..8i+7, 8..15 the V rows; wave w
    // issues instructions w, w + NW, ...  A lane writes chunk position
    // (lane & 7) of tile row 8i + (lane >> 3), so it fetches the logical chunk
    // that the swizzle places there.
#define FMA_ISSUE_TILE(T, ST)                                                                    \
    do {                                                                                         \
        const int t_ = (T), st_ = (ST);                                                          \
        if (t_ < nnear) {                                                                        \
            long long tok0;                                                                      \
            int ux = 0, uy = 0, sub = 0;                                                         \
            if constexpr (GEOM == GEOM_2D) {                                                     \
                const int ci = t_ / tpc;                                                         \
                sub = t_ - ci * tpc;                                                             \
                ux = cx + dx0 + ci / ncy;                                                        \
                uy = cy + dy0 + ci % ncy;                                                        \
                tok0 = 0;                                                                        \
            } else {                                                                             \
                tok0 = klo + (long long)t_ * KT;                                                 \
            }                                                                                    \
            for (int j = wave; j < 16; j += NW) {                                                \
                const int i = j & 7;                                                             \
                const bool isv = j >= 8;                                                         \
                long long tok;                                                                   \
                if constexpr (GEOM == GEOM_2D) {                                                 \
                    const int p0 = sub * KT + 8 * i;                                             \
                    tok = (long long)(ux * r_ + (p0 >> lg_r)) * side_ + uy * r_ + (p0 & (r_ - 1)); \
                } else {                                                                         \
                    tok = tok0 + 8 * i;                                                          \
                }                                                                                \
                const char *src = (isv ? vg : kg) + tok * ROWB + (isv ? ldv : ((i & 1) ? ldk1 : ldk0)); \
                unsigned char *dst = (isv ? sm.v[st_] : sm.k[st_]) + i * 1024;                    \
                __builtin_amdgcn_global_load_lds((gbl_void *)src, (lds_void *)dst, 16, 0, 0);    \
            }                                                                                    \
        } else {                                                                                 \
            const int ct = t_ - nnear;                                                           \
            for (int j = wave; j < 16; j += NW) {                                                \
                const int i = j & 7;                                                             \
                const bool isv = j >= 8;                                                         \
                int row = sm.crow[ct * KT + 8 * i + lrow];                                       \
                row = row < 0 ? 0 : row;                                                         \
                const char *src = (isv ? vbar : kbar) + (long long)row * ROWB +                  \
                                  (isv ? ldv : ((i & 1) ? ldk1 : ldk0)) - lrow * ROWB;           \
                unsigned char *dst = (isv ? sm.v[st_] : sm.k[st_]) + i * 1024;                    \
                __builtin_amdgcn_global_load_lds((gbl_void *)src, (lds_void *)dst, 16, 0, 0);    \
            }                                                                                    \
        }                                                                                        \
    } while (0)
    const int r_ = a.r, side_ = a.side;
    (void)r_;
    (void)side_;

    // ------------------------------------------------ online softmax state
    const float c = a.scale_log2;
    float mrun = -1.0e30f;   // reference maximum (log2 units); finite so exp2 of differences is safe
    float lrun = 0.f;        // this lane's part of the row sum
    f32x16 o0 = {0}, o1 = {0};

    __syncthreads();          // coarse slot table visible
    FMA_ISSUE_TILE(0, 0);
    for (int t = 0; t < ntiles; ++t) {
        const int st = t & (NSTAGE - 1);
        __builtin_amdgcn_s_waitcnt(0);   // this wave's loads of tile t have landed
        __syncthreads();                 // ... and everyone's; tile t-1 is no longer read
        if (t + 1 < ntiles) FMA_ISSUE_TILE(t + 1, (t + 1) & (NSTAGE - 1));

        const bool near = t < nnear;
        int nkb = 2;
        unsigned long long cm = ~0ull;
        long long key0 = 0;
        bool diag = false;
        if (near) {
            if constexpr (GEOM != GEOM_2D) {
                key0 = klo + (long long)t * KT;
                if (a.causal) {
                    if (key0 > wave_q0 + 31) continue;       // every key after this wave's queries
                    diag = key0 + KT - 1 > wave_q0;
                }
            }
        } else {
            const int ct = t - nnear;
            const int left = nslot - ct * KT;
            nkb = left > 32 ? 2 : 1;
            cm = sm.cmask[ct];
        }

        const unsigned char *kt = sm.k[st];
        const unsigned char *vt = sm.v[st];

        // ---- S^T = K Q^T
        f32x16 s[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            s[kb] = f32x16{0};
            if (kb < nkb) {
#pragma unroll
                for (int c4 = 0; c4 < 4; ++c4) {
                    const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(kt + kb * 32 * ROWB + koff[c4]);
                    s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[c4], s[kb], 0, 0, 0);
                }
            }
        }

        // ---- masks (only diagonal causal tiles and coarse tiles have any)
        if (diag) {
            const long long lim = qtok - key0 - 4 * hh;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int kr = kb * 32 + (i >> 2) * 8 + (i & 3);
                    if (kr > lim) s[kb][i] = -INFINITY;
                }
        } else if (!near) {
            const unsigned long long ml = cm >> (4 * hh);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int kr = kb * 32 + (i >> 2) * 8 + (i & 3);
                    if (!((ml >> kr) & 1ull) || kb >= nkb) s[kb][i] = -INFINITY;
                }
        }

        // ---- running maximum, lazily raised
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 16; i += 2) mx = fmaxf(mx, fmaxf(s[kb][i], s[kb][i + 1]));
        mx = max_pair(mx) * c;
        // Each query decides for itself (lanes that keep their reference
        // scale by exp2(0) = 1 exactly), so a row's result never depends on
        // the other rows of the wave.
        const bool raise = mx > mrun + 8.0f;
        if (__builtin_amdgcn_ballot_w64(raise)) {
            const float mnew = raise ? mx : mrun;
            const float corr = fast_exp2(mrun - mnew);
            mrun = mnew;
            lrun *= corr;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                o0[i] *= corr;
                o1[i] *= corr;
            }
        }

        // ---- probabilities, row sum, P^T operand, O^T += V^T P^T
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            if (kb < nkb) {
#pragma unroll
                for (int hf = 0; hf < 2; ++hf) {
                    float p[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        p[e] = fast_exp2(fmaf(s[kb][8 * hf + e], c, -mrun));
                        lrun += p[e];
                    }
                    const uint32_t w0 = pack_bf16(p[0], p[1]), w1 = pack_bf16(p[2], p[3]);
                    const uint32_t w2 = pack_bf16(p[4], p[5]), w3 = pack_bf16(p[6], p[7]);
                    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                    const u32x4 pw = {w0, w1, w2, w3};
                    const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
                    const int kbase = (kb * 32 + hf * 16) * ROWB;
#pragma unroll
                    for (int db = 0; db < 2; ++db) {
                        const s16x4 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                            (lds_s16x4 *)(vt + kbase + voff[db]));
                        const s16x4 r2 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                            (lds_s16x4 *)(vt + kbase + 8 * ROWB + voff[db]));
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
        }
    }

    // ------------------------------------------------ epilogue: O = O^T / l
    const float inv = 1.0f / sum_pair(lrun);
    __bf16 *op = static_cast<__bf16 *>(a.out) + qrow;
#pragma unroll
    for (int db = 0; db < 2; ++db) {
        const f32x16 &o = db == 0 ? o0 : o1;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int d = db * 32 + g * 8 + 4 * hh;
            const uint2 w = make_uint2(pack_bf16(o[4 * g] * inv, o[4 * g + 1] * inv),
                                       pack_bf16(o[4 * g + 2] * inv, o[4 * g + 3] * inv));
            *reinterpret_cast<uint2 *>(op + d) = w;
        }
    }
}

#undef FMA_ISSUE_TILE

template <int GEOM>
hipError_t launch_geom(const AttnArgs &a, hipStream_t st)
{
    const unsigned grid = (unsigned)a.tiles_per_slice * (unsigned)a.nslice;
    switch (a.qtile / 32) {
    case 2: hipLaunchKernelGGL((attend_mfma_kernel<2, GEOM>), dim3(grid), dim3(128), 0, st, a); break;
    case 4: hipLaunchKernelGGL((attend_mfma_kernel<4, GEOM>), dim3(grid), dim3(256), 0, st, a); break;
    case 6: hipLaunchKernelGGL((attend_mfma_kernel<6, GEOM>), dim3(grid), dim3(384), 0, st, a); break;
    case 8: hipLaunchKernelGGL((attend_mfma_kernel<8, GEOM>), dim3(grid), dim3(512), 0, st, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attend_bf16(const AttnArgs &a, int geometry, hipStream_t st)
{
    if (a.nslice == 0 || a.tiles_per_slice == 0) return hipSuccess;
    if (a.nslot > MAX_SLOTS) return hipErrorInvalidValue;
    if (geometry == GEOM_1D) return launch_geom<GEOM_1D>(a, st);
    if (geometry == GEOM_2D) return launch_geom<GEOM_2D>(a, st);
    return launch_geom<GEOM_DENSE>(a, st);
}

}  // namespace fma_dev
