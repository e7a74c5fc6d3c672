/*
 * fma.h -- C ABI of the MI355X (gfx950) Fast Multipole Attention forward pass.
 *
 * Fast Multipole Attention (Kang, Tran & De Sterck, arXiv 2310.11960, Sec. 3)
 * lets every query attend at full resolution to the keys/values of its own
 * base block and the two neighbouring blocks (the near field N(i)), and to
 * learned weighted summaries of progressively larger groups of keys/values
 * farther away (the far field, one list of groups per level).  This library
 * computes that forward pass for Q, K, V of shape [B, H, n, d] on one GPU:
 *
 *   1. coarsening: for every level l = 1 .. L-1 and every group G of length
 *      s_l = r * 2^(l-1) (2D: square of side s_l),
 *          k_bar_G = sum_{j in G} pi^k_l[j - start(G)] * k_j   (Eq. agg1d)
 *          k_bar_S = sum_{(x,y) in S} pi^{k,x}_l[x - x_S] pi^{k,y}_l[y - y_S] k_(x,y)
 *                                                             (Eq. agg2d)
 *      and the same for values with pi^v;
 *   2. fused multilevel attention: for every query i, one softmax over the
 *      scores tau * q_i . k_j of its near-field tokens and tau * q_i . k_bar_G
 *      of its far-field groups, then the matching weighted sum of v_j and
 *      v_bar_G (Eq. fma1d / Eq. fma2d), tau = 1/sqrt(d) by default.
 *
 * Geometry (Sec. 3): r = `block`, L = ceil(log2(n / r)) (1D) or
 * ceil(log2(W / r)) (2D), M_l = ceil(n / s_l) groups at level l (2D: M_l^2
 * squares, row-major u*M_l + v with u the row block).  The interaction list
 * of a base block holds at most 3 groups per level in 1D (2 when causal) and
 * 27 squares per level in 2D.
 *
 * Readings of the paper used here:
 *   - one joint softmax over near tokens and far groups (each group counted
 *     once, no size-dependent bias) by default; `norm = FMA_NORM_PER_LEVEL`
 *     selects the normalisation as printed in Eq. fma1d / Eq. fma2d instead:
 *     the near-field weights sum to 1 and, separately, the weights of each
 *     level's groups (all p representatives of them) sum to 1, and the
 *     per-set results are added;
 *   - causal (1D only): near token j is visible to query i iff j <= i, a far
 *     group iff all of its tokens are <= i;
 *   - 2D token t = x*W + y with x the row; pi^(x) weighs rows, pi^(y) columns;
 *   - when n / r (2D: W / r) is not a power of two the last group of a level
 *     is clipped to the sequence and aggregates only existing tokens;
 *   - coarse level rank p (Sec. 3, "Coarse level rank p"): every level has p
 *     learned basis vectors (2D: p pairs), every group p aggregated keys and
 *     values, and each of the p representatives is a source of its own in the
 *     one softmax.  The kernels see each (level, basis) pair as a "coarse set"
 *     laid out like a level; with p = 1 the sets are the levels.
 *
 * Conventions shared by every entry point:
 *   - Memory: the caller owns every buffer.  Q, K, V and `out` are dense
 *     row-major [B, H, n, d] device arrays of the plan's dtype, 16-byte
 *     aligned; `out` must not overlap an input.  Weights are fp32 device
 *     arrays.  The library never allocates device memory: the caller passes
 *     a device workspace of at least fma_workspace_size() bytes
 *     (fma_forward_static instead uses a static per-GPU buffer of the
 *     library's own, see there).
 *   - Streams: `stream` is a hipStream_t passed as `void *` (NULL = the
 *     default stream), so that the header needs no HIP include.  Work is
 *     enqueued asynchronously; the call returns once it is enqueued.
 *   - Errors: every argument is validated before anything is launched; on
 *     error nothing is written and the status is returned.  A message is
 *     kept per thread for fma_last_error().  Launch failures are reported
 *     as FMA_ERR_HIP.
 *   - Determinism: no atomics; repeated calls give bitwise identical output.
 *   - Thread safety: a plan is immutable after fma_plan() and may be used
 *     from several threads / streams at once with distinct workspaces.
 */
#ifndef FMA_MI355X_H
#define FMA_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FMA_OK = 0,
    FMA_ERR_NULL = 1,         /* a required pointer is NULL */
    FMA_ERR_SHAPE = 2,        /* inconsistent sizes (r does not divide n, wrong L, ...) */
    FMA_ERR_UNSUPPORTED = 3,  /* valid for the method, not implemented by these kernels */
    FMA_ERR_WORKSPACE = 4,    /* workspace missing or too small */
    FMA_ERR_HIP = 5,          /* the HIP runtime reported an error */
    FMA_ERR_HOST_ALLOC = 6,   /* host allocation of the plan failed */
    FMA_ERR_ALIGN = 7,        /* a device pointer is not 16-byte aligned */
    FMA_ERR_ARG = 8           /* other invalid argument (aliasing, bad enum, ...) */
} fma_status_t;

typedef enum {
    FMA_F32 = 0,   /* fp32 inputs/outputs, fp32 MFMA, fp32 accumulation */
    FMA_BF16 = 1   /* bf16 inputs/outputs, bf16 MFMA, fp32 accumulation */
} fma_dtype_t;

typedef enum {
    FMA_NORM_JOINT = 0,      /* one softmax over the near tokens and every far group */
    FMA_NORM_PER_LEVEL = 1   /* printed form: near field and each level normalised on their own */
} fma_norm_t;

typedef struct fma_plan_s *fma_plan_t;   /* opaque, host-side, immutable */

/* Problem description (Sec. 3 statement of the problem). */
typedef struct {
    int32_t struct_size;      /* sizeof(fma_desc_t), or the offset of `rank` or of
                                 `query_downsample` for descriptors without those fields */
    int32_t ndim;             /* 1 (sequences) or 2 (token maps of H rows by W columns) */
    int32_t batch;            /* B >= 0 */
    int32_t heads;            /* H >= 0 */
    int64_t seq_len;          /* n >= 0; 2D: n == H * side, token x * W + y in row x, column y */
    int32_t side;             /* 2D map width W (columns, > 0); H = seq_len / W; ignored (0) in 1D */
    int32_t head_dim;         /* d: 32, 64 or 128 (the matrix-core fused attention and streaming
                                 coarsening are built for 64; 32 and 128 run on the register-
                                 staged attention and the chunk / tile coarsening; the backward
                                 takes 64 only) */
    int32_t block;            /* r: 1D block length / 2D cell side; r | n (2D: r | W and r | H) */
    int32_t num_levels;       /* L = ceil(log2(n/r)) (2D: max(H, W)/r, the longer side); -1 derives it */
    int32_t causal;           /* 0 or 1; 1D only */
    int32_t dtype;            /* fma_dtype_t */
    int32_t weights_per_head; /* 1: weights are [H][wlen]; 0: one [wlen] set for all heads */
    float softmax_scale;      /* tau; 0 selects 1/sqrt(head_dim) */
    int32_t rank;             /* p >= 1 basis vectors per level (Sec. 3); 0 selects 1.  A
                                 struct_size that ends before this field means p = 1 */
    int32_t norm;             /* fma_norm_t; a struct_size that ends before `rank` means joint */
    int32_t query_downsample; /* 1: FMA-linear (queries downsampled on every coarse level; use
                                 fma_forward_linear); 0: FMA.  A struct_size that ends before
                                 this field means 0 */
} fma_desc_t;

/* Validate `desc` and build a plan.  Host memory only.
 * Shapes the method allows but these kernels do not implement return
 * FMA_ERR_UNSUPPORTED: head_dim other than 32, 64 or 128; 1D block other than 16, 32 or a
 * multiple of 64 up to 256; 2D block other than 4, 8 or 16; causal 2D;
 * more than 17 levels;
 * (L-1) * rank above 64 coarse sets, or interaction lists longer than the
 * fused kernel's 448 slots (2D: 27 * (L-1) * rank; per-level normalisation
 * pads each level's 3p (2D: 27p) slots to 4, 8, 16 or 32, and a 2D level of
 * rank p >= 2 to a multiple of 32, so it needs 3p <= 32 in 1D and
 * (L-1) * ceil(27p / 32) * 32 <= 448 in 2D).  rank < 0 or an unknown norm is
 * FMA_ERR_ARG.  FMA-linear plans must be bidirectional, rank 1, joint
 * normalisation (FMA_ERR_UNSUPPORTED otherwise). */
fma_status_t fma_plan(const fma_desc_t *desc, fma_plan_t *out_plan);

/* Release a plan.  NULL is a no-op. */
fma_status_t fma_destroy(fma_plan_t plan);

/* Device workspace the forward/coarsen/attend calls need, in bytes: the
 * coarse keys and values [2][B][H][R][d] in the plan's dtype (K_bar then
 * V_bar; rows ordered by level, then basis, then group: basis s of level l
 * starts at row p * sum_{l'<l} M_l' + s * M_l, 2D with M^2 squares), followed
 * (256-byte aligned) by fp32 partial sums of the split coarsening.  0 when
 * L <= 1. */
fma_status_t fma_workspace_size(fma_plan_t plan, size_t *bytes);

/* Number of fp32 weights per head for each of pi^k and pi^v:
 * 1D: p * sum_l s_l; basis s of level l at offset p*r*(2^(l-1)-1) + s*s_l;
 * 2D: p * sum_l 2*s_l; basis s of level l at offset p*2r*(2^(l-1)-1) + s*2*s_l,
 *     holding pi^(x) then pi^(y). */
fma_status_t fma_weights_len(fma_plan_t plan, int64_t *floats_per_head);

/* Coarse rows per (batch, head): R = p * sum_l M_l (1D) or p * sum_l M_l^2 (2D). */
fma_status_t fma_coarse_rows(fma_plan_t plan, int64_t *rows);

/* Levels L of the plan's hierarchy. */
fma_status_t fma_num_levels(fma_plan_t plan, int32_t *levels);

/* Full 1D forward pass (Eq. agg1d + Eq. fma1d): coarsening, then the fused
 * multilevel attention, both enqueued on `stream`.
 *   q, k, v : [B,H,n,d] device, plan dtype      out : [B,H,n,d] device
 *   wk, wv  : fp32 device, [H][wlen] or [wlen]  (may be NULL when L <= 1)
 *   workspace / workspace_bytes : see fma_workspace_size (NULL/0 when L <= 1)
 * A 2D plan returns FMA_ERR_SHAPE. */
fma_status_t fma_forward_1d(fma_plan_t plan, const void *q, const void *k, const void *v,
                            const float *wk, const float *wv, void *out,
                            void *workspace, size_t workspace_bytes, void *stream);

/* Full 2D forward pass (Eq. agg2d + Eq. fma2d) on a W x W token map stored
 * row-major (token x*W + y).  Arguments as fma_forward_1d; per level the
 * weights hold pi^(x) then pi^(y).  A 1D plan returns FMA_ERR_SHAPE. */
fma_status_t fma_forward_2d(fma_plan_t plan, const void *q, const void *k, const void *v,
                            const float *wk, const float *wv, void *out,
                            void *workspace, size_t workspace_bytes, void *stream);

/* Coarsening alone (Eq. agg1d / Eq. agg2d): writes K_bar and V_bar into
 * the workspace (layout above).  The same kernels the forward pass runs. */
fma_status_t fma_coarsen(fma_plan_t plan, const void *k, const void *v,
                         const float *wk, const float *wv,
                         void *workspace, size_t workspace_bytes, void *stream);

/* Fused multilevel attention alone (Eq. fma1d / Eq. fma2d), reading K_bar
 * and V_bar from a workspace filled by fma_coarsen. */
fma_status_t fma_attend(fma_plan_t plan, const void *q, const void *k, const void *v,
                        const void *workspace, size_t workspace_bytes, void *out, void *stream);

/* Debug export of the interaction lists the fused kernel uses (the groups
 * G_l(i) of Sec. 3, per base block): int32 device array
 * [nblocks][L-1][K] with K = 3 (1D) or 27 (2D), ascending group index
 * (2D: u*My_l + v for the square in row u and column v of level l, which
 * has Mx_l = ceil(H/s_l) rows and My_l = ceil(W/s_l) columns of squares),
 * padded with -1.  Causal plans list only visible groups.  nblocks = n/r
 * (1D) or (H/r)(W/r) (2D, row-major cells). */
fma_status_t fma_interaction_lists(fma_plan_t plan, int32_t *dev_out, void *stream);

/* Dense softmax attention softmax(tau Q K^T) V over the whole sequence (causal
 * when the plan is causal) with the same tiling machinery -- a context
 * baseline for timing, not part of FMA (Sec. 1, Eq. attn). */
fma_status_t fma_dense_reference(fma_plan_t plan, const void *q, const void *k, const void *v,
                                 void *out, void *stream);

/* Test export: the scalar launch parameters the plan hands its kernels, for
 * host-side checks of the kernels' address arithmetic (no device access).
 * Writes *count = 40 + 6 * sets int64 values to out (FMA_ERR_WORKSPACE,
 * with *count set, if capacity is smaller), in this order:
 *   n, side (W), block, cells along x (H/r; 1D: blocks), queries per query tile,
 *   query tiles per slice, slices (B*H), coarse rows per slice R, causal,
 *   list slots per query tile, list slots per level, rank, per-level
 *   normalisation, ndim, bytes per element, heads, weight stride between
 *   heads (0: shared), weights per head, coarse sets;
 *   coarsening: unit (1D) or tile side (2D), rows per thread (fp32 1D),
 *   units (2D: tiles) per slice, tiles along y (2D), first partial set,
 *   partial sets, partial span, partials per (tensor, slice, set), ring
 *   depth of the bf16 streaming kernels (0: fp32 kernels), LDS bytes per
 *   streaming wave, LDS bytes per coarsening workgroup;
 *   workspace: partial-sum offset, coarse bytes, total bytes;
 *   FMA-linear, weight sets (heads or 1), dtype, whether the bf16 fused
 *   attention takes the 2D map's cells in horizontal pairs;
 *   2D: map height H, cells along y (W/r), tiles along x (0 in 1D);
 * then per coarse set: first coarse row, groups (2D: rows of squares),
 * 2D columns of squares (1D: 1), group size, weight offset, level. */
fma_status_t fma_plan_params(fma_plan_t plan, int64_t *out, int32_t capacity, int32_t *count);

/* Achievable-bandwidth reference for the coarsening pass (a bench export,
 * not part of the method): one kernel streams src_bytes of `src` once with
 * 16-byte loads and writes one 16-byte word to `dst` per `write_every` words
 * read (a power of two, 1 .. 256), the read-dominated mix of the coarsening,
 * which reads K and V once and writes 1/40 to 1/60 of that.  dst must hold
 * ceil(src_bytes / 32768) * (2048 / write_every) words of 16 bytes
 * (FMA_ERR_WORKSPACE otherwise); src_bytes a multiple of 16, both 16-byte
 * aligned, not overlapping. */
fma_status_t fma_stream_reference(const void *src, size_t src_bytes, void *dst, size_t dst_bytes,
                                  int32_t write_every, void *stream);

/* FMA-linear forward (query downsampling; the paper's O(n) variant, which it
 * names but does not define -- the reading implemented here): the queries
 * of every level-l group are aggregated with learned weights pi^q (fp32,
 * the layout of wk: [H][wlen] or [wlen]) into a coarse query, and every token
 * of the group scores its level-l far-field groups with that coarse query
 * instead of its own; the near field keeps the token's query; one joint
 * softmax.  1D or 2D (the plan decides); the plan must have
 * query_downsample = 1 (FMA_ERR_ARG otherwise), and fma_forward_1d/2d reject
 * such plans.  Arguments as fma_forward_1d; the workspace
 * (fma_workspace_size of the plan) also holds the coarse queries and, per
 * query block, its far field reduced to (M, Z, U): the maximum score, the sum
 * of 2^(score - M) and the so weighted sum of the coarse values (d + 2 floats). */
fma_status_t fma_forward_linear(fma_plan_t plan, const void *q, const void *k, const void *v,
                                const float *wq, const float *wk, const float *wv, void *out,
                                void *workspace, size_t workspace_bytes, void *stream);

/* Device workspace fma_backward needs, in bytes: the forward's workspace
 * (coarse keys and values, rebuilt by the backward) followed by fp32
 * buffers: the log-sum-exp and rowsum(dO * O) of every query, partial
 * gradients of the coarse rows (2 x slices of a pass x blocks x workgroups
 * per block x list slots x d; one row per query block and workgroup of the
 * query pass),
 * the coarse-row gradients (2 x B*H x R x d) and one dot product per token
 * and coarse set (2 x B*H x sets x n). */
fma_status_t fma_backward_workspace_size(fma_plan_t plan, size_t *bytes);

/* Backward pass of fma_forward_1d / fma_forward_2d (the plan decides which)
 * for training the aggregation weights end to end (Sec. 1, Sec. 3): given
 * the forward's inputs, its output `out` and the upstream gradient `dout`
 * (all [B,H,n,d], plan dtype), writes
 *   dq, dk, dv : [B,H,n,d] plan dtype (overwritten)
 *   dwk, dwv   : fp32, the layout of wk / wv ([H][wlen] or [wlen]); every
 *                (batch, head) slice that uses a weight set adds its part
 * as the gradients of sum(dout * out), under the plan's normalisation
 * (joint, or the printed per-level form of Eq. fma1d / fma2d).  An
 * FMA-linear plan is FMA_ERR_ARG (use fma_backward_linear).  Every block
 * size the forward takes is supported; head_dim must be 64
 * (FMA_ERR_UNSUPPORTED otherwise).  Outputs must not overlap the inputs,
 * each other or the workspace.  Deterministic (no atomics).  The partial
 * gradients are kept for a pass of slices at a time (the plan picks passes
 * of at most 384 MiB of partials), so the workspace stays bounded as B*H
 * grows. */
fma_status_t fma_backward(fma_plan_t plan, const void *q, const void *k, const void *v,
                          const float *wk, const float *wv, const void *out, const void *dout,
                          void *dq, void *dk, void *dv, float *dwk, float *dwv,
                          void *workspace, size_t workspace_bytes, void *stream);

/* Backward pass of fma_forward_linear (FMA-linear plans; the reading of
 * Sec. 3's query downsampling that fma_forward_linear documents): as
 * fma_backward, plus the query weights `wq` (layout of wk) and their
 * gradient `dwq` (fp32, layout of wq, overwritten).  The coarse sources'
 * score gradients reach the coarse queries and, through the query
 * coarsening, q and wq.  dwq must not overlap the inputs, the outputs, the
 * other gradients or the workspace.  A plan that is not FMA-linear is
 * FMA_ERR_ARG (use fma_backward); fma_backward rejects FMA-linear plans the
 * same way.  The workspace is fma_backward_workspace_size bytes.
 * seq_len must stay below 2^31 - 32 and B*H*seq_len/32 below 2^31
 * (FMA_ERR_SHAPE otherwise; the fp32 near-field dq of such a problem would
 * not fit one GPU's memory anyway).  Deterministic (no atomics). */
fma_status_t fma_backward_linear(fma_plan_t plan, const void *q, const void *k, const void *v,
                                 const float *wk, const float *wv, const float *wq, const void *out,
                                 const void *dout, void *dq, void *dk, void *dv, float *dwk, float *dwv,
                                 float *dwq, void *workspace, size_t workspace_bytes, void *stream);

/* Allocation-free full forward pass, for callers that cannot allocate
 * device memory or pass a workspace: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  Computes exactly what
 * fma_forward_1d / fma_forward_2d compute for the plan (1D or 2D, as the plan
 * says; the same kernels), but the workspace (coarse keys and values and the
 * fp32 partial sums, fma_workspace_size bytes) lives in a static buffer of
 * 32 MiB that the library keeps on each GPU it runs on until the process
 * ends.  Plans whose workspace exceeds 32 MiB are rejected with
 * FMA_ERR_WORKSPACE before anything is launched.  Nothing is allocated: no
 * hipMalloc, no hipFree.  The buffer's device address is looked up on the
 * first call on each device (the current device; `stream` must belong to
 * it).  Every call on one GPU shares that GPU's buffer, which keeps the last
 * call's contents (every byte a call reads was written by the same call):
 * calls that overlap on one GPU -- on different streams, or from several
 * threads without ordering -- race on it and must be serialised by the
 * caller.  Other arguments and errors as fma_forward_1d; FMA-linear plans
 * return FMA_ERR_ARG. */
fma_status_t fma_forward_static(fma_plan_t plan, const void *q, const void *k, const void *v,
                                const float *wk, const float *wv, void *out, void *stream);

/* Message of the last failed call on this thread ("" if none). */
const char *fma_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FMA_MI355X_H */
