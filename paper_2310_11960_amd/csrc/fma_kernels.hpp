// fma_kernels.hpp -- kernel argument blocks and launchers (internal to the library).
#pragma once

#include <hip/hip_runtime.h>

#include "fma_device.hpp"

namespace fma_dev {

struct CoarsenArgs {
    const void *k;
    const void *v;
    const float *wk;
    const float *wv;
    void *coarse;          // workspace: [2][nslice][R][d] (K_bar, then V_bar)
    float *part;           // fp32 partials [2][nslice][npartial][part_count][d]
    long long n;           // tokens per slice
    int side;              // 2D map width W (columns; token x * W + y)
    int height;            // 2D map height H (rows)
    int r;                 // base block / cell side
    int head_dim;          // d: 32, 64 or 128 (the streaming kernels: 64 only)
    int two_d;             // 0: 1D chunks, 1: 2D tiles
    int nslice;            // B * H
    int heads;
    long long w_stride;    // floats between heads' weights (0 = shared)
    int R;                 // coarse rows per slice
    int chunk;             // 1D: tokens per unit (bf16) or per workgroup (fp32); 2D: tile side (32)
    int run;               // 1D: rows per thread (CH / 32)
    int nchunk;            // chunks (2D: tiles) per slice
    int tiles_x, tiles_y;  // 2D only: 32x32 tiles along x (rows) and y (columns)
    int first_partial;     // first level (0-based) whose groups span several partial spans
    int npartial;          // levels from first_partial on
    int part_span;         // rows (2D: tile side) one partial covers
    int part_count;        // partials per (tensor, slice, level)
    int depth;             // 1D bf16 (matrix-core streaming kernel): ring slots per wave; 0: fp32 kernel
    int wave_lds;          // 1D bf16: LDS bytes per wave (ring, zeros, output staging)
    Levels lv;
};

struct AttnArgs {
    const void *q;
    const void *k;
    const void *v;
    const void *kbar;      // coarse keys   [nslice][R][d]
    const void *vbar;      // coarse values [nslice][R][d]
    void *out;
    long long n;           // tokens per slice
    int side;              // 2D map width W (columns; token x * W + y)
    int r;                 // base block (1D) / cell side (2D)
    int head_dim;          // d: 32, 64 or 128 (the bf16 matrix-core kernels: 64 only)
    int nbx, nby;          // 2D cells along x (rows, H / r) and y (columns, W / r); cell cx * nby + cy
    int qtile;             // queries per workgroup
    int tiles_per_slice;   // query tiles per slice
    int nslice;
    int R;
    int causal;
    int ncoarse_tiles;     // 64-row tiles of interaction-list slots
    int nslot;             // interaction-list slots: (L-1) * slot_group
    int slot_group;        // slots per level: K * rank (joint) or K * rank rounded up to 4, 8, 16 or 32
                           // (per-level normalisation), K = 3 (1D) or 27 (2D); slot
                           // l * slot_group + b * K + j is entry j of basis b of level l+1
    int rank;              // basis vectors per level
    int norm_level;        // 1: printed per-level normalisation (FMA_NORM_PER_LEVEL)
    const void *qbar;      // FMA-linear: coarse queries [nslice][R][d] (nullptr: FMA)
    float *lin_far;        // FMA-linear, bf16: per query block (M, Z, U[d]) of the far field [blocks][d + 2]
    long long lin_far_elems;
    float scale_log2;      // softmax scale * log2(e)
    Levels lv;
};

// Backward pass (gradients of sum(dO * O)).  Every buffer comes with its
// size in elements; the kernels check each global access against it.
struct BwdArgs {
    const void *q, *k, *v, *out, *dout;   // [S][n][64] I/O dtype
    const void *kbar, *vbar;              // coarse keys / values [S][R][64] I/O dtype
    const float *wk, *wv;                 // weights [heads_w][wlen]
    void *dq, *dk, *dv;                   // [S][n][64] I/O dtype
    float *dwk, *dwv;                     // weight gradients [heads_w][wlen]
    float *lse;                           // [S][n] log2-domain log-sum-exp of the scaled scores
    float *delta;                         // [S][n] rowsum(dO * O)
    float *part;                          // [2][pslices][npart][nslot][64] per-workgroup dK_bar, dV_bar
                                          // partials of the slices of one pass
    float *dkbar, *dvbar;                 // [S][R][64]
    float *dotk, *dotv;                   // [S][nsets][n] k_t . dK_bar (v_t . dV_bar) of each token's group
    // FMA-linear (reading R18): coarse queries and the query-side gradients
    const void *qbar;                     // [S][R][64] I/O dtype (nullptr: FMA)
    const float *wq;                      // query weights [heads_w][wlen]
    float *dwq;                           // their gradient
    float *qpart;                         // [S][npart][nsets][64] per-workgroup dQ_bar partials
    float *dqbar;                         // [S][R][64]
    float *dqn;                           // [S][n][64] the near field's part of dq, fp32
    float *dotq;                          // [S][nsets][n] q_t . dQ_bar of each token's group
    long long qpart_elems, dqn_elems;
    int wsets;            // weight tensors the weight-gradient kernels process (2: k and v)
    long long n;          // tokens per slice
    int side, r;          // 2D map width W, block / cell side
    int height;           // 2D map height H (rows)
    int nbx, nby;         // 2D cells along x (H / r) and y (W / r); cell cx * nby + cy
    int qtile;            // tokens per block (r in 1D, r*r in 2D)
    int nblocks;          // blocks per slice
    int npart;            // coarse-partial rows per slice: one per (query block, workgroup of the
                          // query pass); set by the backward launcher
    int nslice, heads, heads_w;
    int slice0, pslices;  // the query pass and its reduction run over slices [slice0, slice0 + pslices)
                          // at a time, so that the partials need pslices slices of space
    int R, causal, nslot, rank;
    int norm_level;       // 1: printed per-level normalisation (FMA_NORM_PER_LEVEL)
    int slot_group;       // list slots per level (per-level: 3p or 27p padded to 4 .. 32)
    long long w_stride;   // floats between heads' weights (0 = shared)
    int wlen;
    float scale, scale_log2;
    long long io_elems, coarse_elems, part_elems, dot_elems, lse_elems, w_elems;
    Levels lv;
};

enum Geometry { GEOM_1D = 0, GEOM_2D = 1, GEOM_DENSE = 2, GEOM_2DP = 3 /* 2D, cells in pairs (bf16 kernel) */ };

// Resident workgroups of `kernel` (threads per workgroup, dynamic LDS bytes)
// on the whole current device: CU count x occupancy per CU.  Looked up once
// per (device, kernel, threads, LDS) and kept; thread-safe.  0 on failure
// (nothing is kept then).
int resident_slots(const void *kernel, int threads, size_t smem);

hipError_t launch_coarsen(const CoarsenArgs &a, bool bf16, size_t smem_bytes, hipStream_t st);
hipError_t launch_attend(const AttnArgs &a, bool bf16, int geometry, hipStream_t st);
hipError_t launch_attend_bf16(const AttnArgs &a, int geometry, hipStream_t st);
hipError_t launch_lin_far(const AttnArgs &a, int geometry, hipStream_t st);
hipError_t launch_lists(int two_d, int nblocks, int nby, int causal, const Levels &lv,
                        int32_t *out, hipStream_t st);
hipError_t launch_backward(const BwdArgs &a, bool bf16, bool two_d, hipStream_t st);
hipError_t launch_stream_ref(const void *src, long long nwords, void *dst, long long ndst, int write_every,
                             hipStream_t st);
long long stream_ref_dst_words(long long nwords, int write_every);

}  // namespace fma_dev
