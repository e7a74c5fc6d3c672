// fma_api.hip -- the C ABI declared in include/fma.h: plan validation,
// geometry, workspace sizing and the launch sequence on the caller's stream.
// Host code only; the kernels live in coarsen.hip, attend.hip and lists.hip.
#include <math.h>
#include <stddef.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <new>

#include "fma.h"
#include "fma_kernels.hpp"

using fma_dev::Levels;

// Occupancy cache behind fma_dev::resident_slots: a small table guarded by a
// mutex; an entry is added only after a successful query.
int fma_dev::resident_slots(const void *kernel, int threads, size_t smem)
{
    struct Entry {
        const void *kernel;
        int dev, threads;
        size_t smem;
        int slots;
    };
    static std::mutex mu;
    static Entry table[256];
    static int used = 0;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
    std::lock_guard<std::mutex> lock(mu);
    for (int i = 0; i < used; ++i)
        if (table[i].kernel == kernel && table[i].dev == dev && table[i].threads == threads && table[i].smem == smem)
            return table[i].slots;
    int cus = 0, per = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, threads, smem) != hipSuccess) return 0;
    const int slots = cus * (per > 0 ? per : 1);
    if (used < 256) table[used++] = Entry{kernel, dev, threads, smem, slots};
    return slots;
}

struct fma_plan_s {
    fma_desc_t desc;
    int L;                 // levels of the hierarchy
    long long n;           // tokens per slice
    int W;                 // 2D width (columns)
    int H;                 // 2D height (rows, seq_len / W)
    int r;                 // block
    int nslice;            // B * H
    int nbx;               // 2D cells along x, H / r (1D: blocks)
    int nby;               // 2D cells along y, W / r (1D: 1)
    int nblocks;           // query tiles per slice (blocks / cells)
    long long R;           // coarse rows per slice
    long long wlen;        // weight floats per head
    int esize;             // bytes per element
    int rank;              // p: basis vectors per level
    int norm_level;        // 1: per-level normalisation
    int linear;            // 1: FMA-linear (query downsampling)
    size_t lin_q_offset;   // FMA-linear: the query coarsening's workspace (coarse queries first)
    size_t lin_far_offset; // FMA-linear: per query block (M, Z, U[d]) of the far field (bf16 plans)
    int slot_group;        // interaction-list slots per level (see AttnArgs)
    int nslot;             // interaction-list slots per query block
    float scale;
    Levels lv;             // coarse sets (level, basis), what the kernels walk
    Levels rlv;            // the levels alone (one set per level), for the list export
    // coarsening decomposition
    int chunk, run, nchunk, tiles_x, tiles_y, first_partial, npartial;
    int depth;             // 1D bf16 coarsening: ring slots per wave (0: fp32 kernel)
    int small;             // blocks smaller than a wave (1D r < 64, 2D r < 8): register-staged attention
    int d;                 // head dim (32, 64 or 128)
    int generic;           // register-staged attention and chunk / tile coarsening: small blocks, fp32
                           // (coarsening), or d != 64 (the matrix-core kernels are built for 64)
    int wave_lds;          // 1D bf16 coarsening: LDS bytes per wave
    int part_span;         // rows (2D: tile side) covered by one coarsening partial sum
    int part_count;        // partial sums per (tensor, slice, level)
    size_t coarsen_smem;
    size_t coarse_bytes, part_offset, part_bytes, ws_bytes;
    // backward workspace: the forward's, then lse, D, coarse partials,
    // dK_bar / dV_bar and the weight-gradient dot products (256-byte aligned)
    int npart_max;         // backward: coarse-partial rows per slice, one per (query block, workgroup)
    int bw_pslices;        // backward: slices per pass of the query pass and its reduction
    size_t bw_part_floats; // backward: floats of the partials' space
    size_t bw_lse, bw_delta, bw_part, bw_cbar, bw_dot, bw_bytes;
    // FMA-linear backward: dQ_bar partials, dQ_bar, the near field's dq (fp32), q . dQ_bar
    size_t bw_qpart, bw_dqbar, bw_dqn, bw_dotq;
};

namespace {

thread_local char g_err[512];

fma_status_t fail(fma_status_t st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return st;
}

fma_status_t ok()
{
    g_err[0] = 0;
    return FMA_OK;
}

int levels_for(long long ratio)
{
    int L = 0;
    long long p = 1;
    while (p < ratio) {
        p *= 2;
        ++L;
    }
    return L;
}

long long cdiv(long long a, long long b) { return (a + b - 1) / b; }

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool overlap(const void *a, size_t na, const void *b, size_t nb)
{
    if (!a || !b || na == 0 || nb == 0) return false;
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + nb && y < x + na;
}

// Pick the 1D chunk CH = r * 2^k: a thread's run of CH/NRUN rows (NRUN =
// 2048 / d runs: d / 8 threads per row) must be a multiple of 4 and divide r
// (so a run stays inside one base block); the weight windows plus the
// reduction buffers must fit in 64 KB of LDS; the largest such chunk (up to
// 1024 tokens) that still gives >= 1024 workgroups is used, else the smallest.
void choose_chunk_1d(fma_plan_s *p)
{
    int best = -1, smallest = -1;
    size_t best_smem = 0, small_smem = 0;
    const int nrun = 2048 / p->d;
    for (int k = 5; k >= 0; --k) {
        const long long CH = (long long)p->r << k;
        if (CH % nrun || CH > 1024) continue;
        const long long run = CH / nrun;
        if (run % 4 || p->r % run) continue;
        long long wfl = 0;   // weight window of the widest pass
        for (int v0 = 0; v0 < p->lv.nlev; v0 += fma_dev::kPassSets) {
            long long w = 0;
            for (int l = v0; l < p->lv.nlev && l < v0 + fma_dev::kPassSets; ++l)
                w += p->lv.size[l] < CH ? p->lv.size[l] : CH;
            wfl = w > wfl ? w : wfl;
        }
        const size_t smem = (size_t)wfl * 4 + 2 * 32 * 64 * 4;
        if (smem > 65536) continue;
        smallest = (int)CH;
        small_smem = smem;
        if (best < 0 && 2LL * p->nslice * cdiv(p->n, CH) >= 1024) {
            best = (int)CH;
            best_smem = smem;
        }
    }
    if (best < 0) {
        best = smallest;
        best_smem = small_smem;
    }
    p->chunk = best;
    p->coarsen_smem = best_smem;
}

// 1D bf16 coarsening on the matrix cores (coarsen1d_stream): every wave
// streams units of CW tokens through a ring of D slots; a slot holds 16 rows
// (2 KB) and the rows' weights of up to 4 * NWD coarse sets (256 B per four
// sets).  A pass builds at most 32 sets (rank * (L - 1) <= 32 is one pass);
// the LDS is sized for the widest pass.  Each wave also keeps 64 zero bytes,
// stages its closed rows (16 bf16 rows, written out whenever full) and its
// partial rows of the sets wider than CW (8 fp32 rows at a time).
// D is the depth that keeps the most bytes in flight per CU (160 KB of LDS
// per CU, at most 80 KB per workgroup of four waves; on ties the shallower
// ring, i.e. more waves, wins).  CW = r * 2^k, at most 8r and 1024 tokens:
// the largest that still gives every wave resident at that depth a unit;
// the smallest (r) if none does.
bool choose_stream_1d(fma_plan_s *p)
{
    const int nsets = p->lv.nlev;
    const int npass_sets = nsets < fma_dev::kStreamSets ? nsets : fma_dev::kStreamSets;
    const int nwd = fma_dev::stream_weight_loads(npass_sets);
    if (nwd == 0) return false;
    if (p->wlen >= (1LL << 29)) return false;                              // 32-bit weight byte offsets
    if (2LL * p->nslice * p->R >= (1LL << 31)) return false;               // 32-bit output row indices
    long long best_inflight = -1, best_lds = 0, best_wgs = 0;
    int best_d = 0;
    for (int D = 2; D <= 6; ++D) {
        const long long wl = fma_dev::stream_wave_lds(D, nwd);
        if (4 * wl > 81920) continue;
        long long wgs = 163840 / (4 * wl);
        if (wgs > 6) wgs = 6;
        const long long inflight = wgs * 4 * D * 2048;
        if (inflight > best_inflight) {
            best_inflight = inflight;
            best_d = D;
            best_lds = wl;
            best_wgs = wgs;
        }
    }
    if (best_d == 0) return false;
    // the widest unit that still gives every resident wave one
    long long cw = p->r;
    for (int k = 3; k >= 0; --k) {
        const long long c = (long long)p->r << k;
        if (c > 1024) continue;
        if (2LL * p->nslice * cdiv(p->n, c) >= 256 * 4 * best_wgs) {
            cw = c;
            break;
        }
    }
    p->chunk = (int)cw;
    p->depth = best_d;
    p->wave_lds = (int)best_lds;
    p->coarsen_smem = (size_t)(4 * best_lds);
    return true;
}

// 2D bf16 coarsening on the matrix cores (coarsen2d_stream): units are the
// 32x32-pixel tiles; a pass holds consecutive sets of at most 32 columns in
// all (stream2d_cols).  NWY follows the largest pass's set count; D (2 .. 4)
// is the depth that keeps the most bytes in flight per CU, at most 80 KB of
// LDS per workgroup of four waves (ties: the shallower ring).
bool choose_stream_2d(fma_plan_s *p)
{
    if (p->W % 32 || p->H % 32) return false;
    if (p->wlen >= (1LL << 29)) return false;                              // 32-bit weight byte offsets
    if (2LL * p->nslice * p->R >= (1LL << 31)) return false;               // 32-bit output row indices
    int most_sets = 0;
    for (int v0 = 0; v0 < p->lv.nlev;) {
        int cols = 0, v1 = v0;
        while (v1 < p->lv.nlev && cols + fma_dev::stream2d_cols(p->lv.size[v1]) <= 32)
            cols += fma_dev::stream2d_cols(p->lv.size[v1++]);
        most_sets = v1 - v0 > most_sets ? v1 - v0 : most_sets;
        v0 = v1;
    }
    const int nwy = fma_dev::stream2d_weight_loads(most_sets);
    if (nwy == 0) return false;
    long long best_inflight = -1, best_lds = 0;
    int best_d = 0;
    for (int D = 2; D <= 4; ++D) {
        const long long wl = fma_dev::stream2d_wave_lds(D, nwy);
        if (4 * wl > 81920) continue;
        long long wgs = 163840 / (4 * wl);
        if (wgs > 6) wgs = 6;
        const long long inflight = wgs * 4 * D * 2048;
        if (inflight > best_inflight) {
            best_inflight = inflight;
            best_d = D;
            best_lds = wl;
        }
    }
    if (best_d == 0) return false;
    p->depth = best_d;
    p->wave_lds = (int)best_lds;
    p->coarsen_smem = (size_t)(4 * best_lds);
    return true;
}

}  // namespace

extern "C" {

const char *fma_last_error(void) { return g_err; }

fma_status_t fma_plan(const fma_desc_t *d, fma_plan_t *out)
{
    if (!d || !out) return fail(FMA_ERR_NULL, "fma_plan: desc and out_plan must not be NULL");
    *out = nullptr;
    // descriptors written before the rank / query_downsample fields existed
    // are accepted as rank 1, joint normalisation / FMA
    const bool full = d->struct_size == (int32_t)sizeof(fma_desc_t);
    const bool has_rank = full || d->struct_size == (int32_t)offsetof(fma_desc_t, query_downsample);
    if (!has_rank && d->struct_size != (int32_t)offsetof(fma_desc_t, rank))
        return fail(FMA_ERR_ARG, "fma_plan: struct_size %d != sizeof(fma_desc_t) %zu", d->struct_size,
                    sizeof(fma_desc_t));
    const int linear = full ? d->query_downsample : 0;
    if (linear != 0 && linear != 1) return fail(FMA_ERR_ARG, "fma_plan: query_downsample must be 0 or 1");
    const int rank = has_rank ? (d->rank == 0 ? 1 : d->rank) : 1;
    if (rank < 1) return fail(FMA_ERR_ARG, "fma_plan: rank must be >= 1 (0 selects 1), got %d", d->rank);
    const int norm = has_rank ? d->norm : FMA_NORM_JOINT;
    if (norm != FMA_NORM_JOINT && norm != FMA_NORM_PER_LEVEL)
        return fail(FMA_ERR_ARG, "fma_plan: unknown norm %d", norm);
    if (d->ndim != 1 && d->ndim != 2) return fail(FMA_ERR_ARG, "fma_plan: ndim must be 1 or 2, got %d", d->ndim);
    if (d->dtype != FMA_F32 && d->dtype != FMA_BF16)
        return fail(FMA_ERR_ARG, "fma_plan: unknown dtype %d", d->dtype);
    if (d->batch < 0 || d->heads < 0 || d->seq_len < 0)
        return fail(FMA_ERR_SHAPE, "fma_plan: negative batch/heads/seq_len");
    if (d->block <= 0) return fail(FMA_ERR_SHAPE, "fma_plan: block must be positive, got %d", d->block);
    if (d->head_dim != 32 && d->head_dim != 64 && d->head_dim != 128)
        return fail(FMA_ERR_UNSUPPORTED, "fma_plan: head_dim %d not implemented (32, 64 or 128)", d->head_dim);
    if (d->causal != 0 && d->causal != 1) return fail(FMA_ERR_ARG, "fma_plan: causal must be 0 or 1");
    if (d->weights_per_head != 0 && d->weights_per_head != 1)
        return fail(FMA_ERR_ARG, "fma_plan: weights_per_head must be 0 or 1");
    if (!isfinite(d->softmax_scale)) return fail(FMA_ERR_ARG, "fma_plan: softmax_scale is not finite");
    if ((long long)d->batch * d->heads > 0x7fffffffLL) return fail(FMA_ERR_SHAPE, "fma_plan: B*H too large");

    fma_plan_s p;
    memset(&p, 0, sizeof(p));
    memcpy(&p.desc, d, full ? sizeof(fma_desc_t) : has_rank ? offsetof(fma_desc_t, query_downsample)
                                                        : offsetof(fma_desc_t, rank));
    p.desc.struct_size = (int32_t)sizeof(fma_desc_t);
    p.desc.rank = rank;
    p.desc.norm = norm;
    p.desc.query_downsample = linear;
    p.rank = rank;
    p.norm_level = norm == FMA_NORM_PER_LEVEL;
    p.linear = linear;
    if (linear && (d->causal || rank != 1 || p.norm_level))
        return fail(FMA_ERR_UNSUPPORTED,
                    "fma_plan: FMA-linear is bidirectional, rank 1, joint normalisation (a group's coarse query "
                    "mixes the queries of later tokens, so causal use is not defined)");
    p.n = d->seq_len;
    p.r = d->block;
    p.nslice = d->batch * d->heads;
    p.esize = d->dtype == FMA_BF16 ? 2 : 4;
    p.scale = d->softmax_scale != 0.f ? d->softmax_scale : 1.0f / sqrtf((float)d->head_dim);

    long long ratio;
    if (d->ndim == 1) {
        if (p.n % p.r) return fail(FMA_ERR_SHAPE, "fma_plan: block %d does not divide seq_len %lld", p.r, p.n);
        if ((p.r % 64 || p.r > 256) && p.r != 16 && p.r != 32)
            return fail(FMA_ERR_UNSUPPORTED,
                        "fma_plan: 1D block %d not implemented (16, 32 or a multiple of 64 up to 256)", p.r);
        p.small = p.r < 64;
        ratio = p.n / p.r;
        p.nbx = (int)ratio;
        p.nby = 1;
        p.nblocks = (int)ratio;
        p.W = 0;
        p.H = 0;
    } else {
        if (d->causal) return fail(FMA_ERR_UNSUPPORTED, "fma_plan: causal 2D attention is not defined");
        // an H x W map, H = seq_len / side rows of `side` tokens (reading:
        // the depth follows the longer side)
        if (d->side <= 0 || p.n % d->side || p.n / d->side > 0x7fffffffLL)
            return fail(FMA_ERR_SHAPE, "fma_plan: 2D needs seq_len == H * side (side %d, seq_len %lld)", d->side, p.n);
        p.W = d->side;
        p.H = (int)(p.n / d->side);
        if (p.W % p.r || p.H % p.r)
            return fail(FMA_ERR_SHAPE, "fma_plan: block %d does not divide the %d x %d map", p.r, p.H, p.W);
        if (p.r != 4 && p.r != 8 && p.r != 16)
            return fail(FMA_ERR_UNSUPPORTED, "fma_plan: 2D cell side %d not implemented (4, 8 or 16)", p.r);
        p.small = p.r < 8;
        p.nbx = p.H / p.r;
        p.nby = p.W / p.r;
        if ((long long)p.nbx * p.nby > 0x7fffffffLL) return fail(FMA_ERR_SHAPE, "fma_plan: map too large");
        p.nblocks = p.nbx * p.nby;
        ratio = p.nbx > p.nby ? p.nbx : p.nby;
    }
    if (ratio > (1LL << 30)) return fail(FMA_ERR_SHAPE, "fma_plan: sequence too long");
    p.d = d->head_dim;
    p.generic = p.small || p.d != fma_dev::kHeadDim;
    p.L = levels_for(ratio);
    if (d->num_levels != -1 && d->num_levels != p.L)
        return fail(FMA_ERR_SHAPE, "fma_plan: num_levels %d != ceil(log2(%lld)) = %d", d->num_levels, ratio, p.L);
    const int nlev_real = p.L > 1 ? p.L - 1 : 0;
    if (nlev_real > fma_dev::kMaxCoarse)
        return fail(FMA_ERR_UNSUPPORTED, "fma_plan: %d levels exceed the supported %d", p.L, fma_dev::kMaxCoarse + 1);
    // coarse sets: every (level, basis) pair, level-major (Sec. 3, coarse level rank p)
    const long long nsets_ll = (long long)nlev_real * rank;
    if (nsets_ll > fma_dev::kMaxSets)
        return fail(FMA_ERR_UNSUPPORTED, "fma_plan: %d levels x rank %d exceed the supported %d coarse sets",
                    nlev_real, rank, fma_dev::kMaxSets);
    {
        // interaction-list slots per level: K per basis, padded under
        // per-level normalisation to a power of two up to 32, so that a
        // level's slots form one aligned group of the kernels' 32-key blocks,
        // or (2D, rank >= 2: 27p > 32) to a multiple of 32, so that a level
        // fills whole blocks, which the kernels normalise online
        const long long per = (long long)(d->ndim == 1 ? fma_dev::kSlots1D : fma_dev::kSlots2D) * rank;
        long long grp = per;
        if (p.norm_level) {
            grp = 4;
            while (grp < per && grp < 32) grp *= 2;
            if (grp < per) {
                if (d->ndim == 1)
                    return fail(FMA_ERR_UNSUPPORTED,
                                "fma_plan: 1D per-level normalisation supports at most 32 list slots per level "
                                "(rank <= 10); rank %d needs %lld", rank, per);
                grp = (per + 31) / 32 * 32;
            }
        }
        if (grp * nlev_real > 448)
            return fail(FMA_ERR_UNSUPPORTED, "fma_plan: %d levels x %lld list slots exceed the supported 448",
                        nlev_real, grp);
        p.slot_group = (int)grp;
        p.nslot = (int)(grp * nlev_real);
    }
    const int nlev = (int)nsets_ll;

    p.lv.nlev = nlev;
    p.rlv.nlev = nlev_real;
    long long off = 0, woff = 0;
    const long long span = d->ndim == 1 ? p.n : p.H;
    for (int l = 0; l < nlev_real; ++l) {
        const long long s = (long long)p.r << l;
        const long long M = cdiv(span, s);                      // 2D: rows of squares
        const long long My = d->ndim == 1 ? 1 : cdiv(p.W, s);   // 2D: columns of squares
        p.rlv.size[l] = (int)s;
        p.rlv.M[l] = (int)M;
        p.rlv.My[l] = (int)My;
        p.rlv.lvl[l] = l + 1;
        p.rlv.off[l] = (int)off;
        p.rlv.woff[l] = (int)woff;
        for (int b = 0; b < rank; ++b) {
            const int e = l * rank + b;
            p.lv.size[e] = (int)s;
            p.lv.M[e] = (int)M;
            p.lv.My[e] = (int)My;
            p.lv.lvl[e] = l + 1;
            p.lv.off[e] = (int)off;
            p.lv.woff[e] = (int)woff;
            off += M * My;
            woff += d->ndim == 1 ? s : 2 * s;
        }
    }
    if (off > 0x7fffffffLL || woff > 0x7fffffffLL) return fail(FMA_ERR_SHAPE, "fma_plan: hierarchy too large");
    p.R = off;
    p.wlen = woff;

    if (nlev > 0 && p.nslice > 0) {
        if (d->ndim == 1) {
            if (d->dtype == FMA_BF16 && !p.generic) {
                if (!choose_stream_1d(&p))
                    return fail(FMA_ERR_UNSUPPORTED, "fma_plan: no coarsening decomposition for block %d", p.r);
            } else {
                choose_chunk_1d(&p);
                if (p.chunk <= 0)
                    return fail(FMA_ERR_UNSUPPORTED, "fma_plan: no coarsening decomposition for block %d", p.r);
                p.run = p.chunk / (2048 / p.d);   // rows per thread: 2048 / d runs of a chunk
            }
            p.nchunk = (int)cdiv(p.n, p.chunk);
        } else {
            p.chunk = 32;
            p.run = 0;
            p.tiles_x = (int)cdiv(p.H, 32);
            p.tiles_y = (int)cdiv(p.W, 32);
            p.nchunk = p.tiles_x * p.tiles_y;
            long long wfl = 0;   // weight windows of the widest pass
            for (int v0 = 0; v0 < nlev; v0 += fma_dev::kPassSets) {
                long long w = 0;
                for (int l = v0; l < nlev && l < v0 + fma_dev::kPassSets; ++l)
                    w += 2LL * (p.lv.size[l] < 32 ? p.lv.size[l] : 32);
                wfl = w > wfl ? w : wfl;
            }
            // the tile kernel's two reduction buffers: NT / (d / 8) runs of d channels
            const int nt = fma_dev::coarsen2d_threads(p.r, p.d);
            p.coarsen_smem = (size_t)wfl * 4 + 2 * (size_t)nt * 8 * 4;
            // bf16: the matrix-core streaming kernel where it applies (it
            // sets depth > 0 and its own LDS size)
            if (d->dtype == FMA_BF16 && !p.generic) choose_stream_2d(&p);
        }
        // one partial sum per chunk (2D: per 32x32 tile) for the levels whose
        // groups span several chunks
        p.part_span = p.chunk;
        p.part_count = p.nchunk;
        p.first_partial = nlev;
        for (int l = 0; l < nlev; ++l)
            if (p.lv.size[l] > p.part_span) {
                p.first_partial = l;
                break;
            }
        p.npartial = nlev - p.first_partial;
    }
    p.coarse_bytes = (size_t)2 * p.nslice * p.R * p.d * p.esize;
    p.part_offset = (p.coarse_bytes + 255) & ~(size_t)255;
    p.part_bytes = (size_t)2 * p.nslice * p.npartial * p.part_count * p.d * sizeof(float);
    p.ws_bytes = nlev > 0 ? p.part_offset + p.part_bytes : 0;
    // FMA-linear: a second coarsening workspace of the same shape for the queries
    p.lin_q_offset = (p.ws_bytes + 255) & ~(size_t)255;
    if (p.linear && nlev > 0) {
        p.ws_bytes = p.lin_q_offset + p.ws_bytes;
        p.lin_far_offset = (p.ws_bytes + 255) & ~(size_t)255;
        p.ws_bytes = p.lin_far_offset + (size_t)p.nslice * p.nblocks * (p.d + 2) * sizeof(float);
    }

    {
        auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
        const size_t sn = (size_t)p.nslice * (size_t)p.n;
        // the backward's query pass runs four waves of 32 queries per
        // workgroup (bf16 blocks of a multiple of 128 queries) or two, and
        // stores one partial row per (block, workgroup)
        const long long qtile = d->ndim == 1 ? p.r : (long long)p.r * p.r;
        const int bw_nw = d->dtype == FMA_BF16 && qtile % 128 == 0 ? 4 : 2;
        p.npart_max = (int)((long long)p.nblocks * (((qtile + 31) / 32 + bw_nw - 1) / bw_nw));
        p.bw_lse = up(p.ws_bytes);
        p.bw_delta = up(p.bw_lse + sn * 4);
        p.bw_part = up(p.bw_delta + sn * 4);
        // the partials of one pass of slices: when all slices' partials
        // exceed 384 MiB, the slices run in the fewest equal passes that fit
        // it (at least one slice a pass), so that the workspace does not grow
        // with a partial row per slice of the whole batch; the 2D weight
        // gradients' line sums reuse the space
        const size_t per_slice = nlev > 0 ? (size_t)2 * p.npart_max * p.nslot * fma_dev::kHeadDim : 0;
        const size_t budget = (size_t)384 << 18;   // floats
        p.bw_pslices = p.nslice > 0 ? p.nslice : 1;
        if (per_slice > 0 && (size_t)p.bw_pslices * per_slice > budget) {
            const size_t fit = budget / per_slice > 0 ? budget / per_slice : 1;
            const size_t passes = ((size_t)p.bw_pslices + fit - 1) / fit;
            p.bw_pslices = (int)(((size_t)p.bw_pslices + passes - 1) / passes);
        }
        size_t part_floats = (size_t)p.bw_pslices * per_slice;
        if (d->ndim == 2 && nlev > 0) {
            const size_t lines = (size_t)2 * p.nslice * nlev * 2 * (size_t)(p.H > p.W ? p.H : p.W);
            part_floats = lines > part_floats ? lines : part_floats;
        }
        p.bw_part_floats = part_floats;
        p.bw_cbar = up(p.bw_part + part_floats * 4);
        const size_t cbar = (size_t)2 * p.nslice * p.R * fma_dev::kHeadDim * 4;
        p.bw_dot = up(p.bw_cbar + cbar);
        p.bw_bytes = up(p.bw_dot + (size_t)2 * nlev * sn * 4);
        if (p.linear) {
            p.bw_qpart = p.bw_bytes;
            p.bw_dqbar = up(p.bw_qpart + (size_t)p.nslice * p.npart_max * nlev * fma_dev::kHeadDim * 4);
            p.bw_dqn = up(p.bw_dqbar + (size_t)p.nslice * p.R * fma_dev::kHeadDim * 4);
            p.bw_dotq = up(p.bw_dqn + sn * fma_dev::kHeadDim * 4);
            p.bw_bytes = up(p.bw_dotq + (size_t)nlev * sn * 4);
        }
    }

    fma_plan_s *h = new (std::nothrow) fma_plan_s(p);
    if (!h) return fail(FMA_ERR_HOST_ALLOC, "fma_plan: out of host memory");
    *out = h;
    return ok();
}

fma_status_t fma_destroy(fma_plan_t plan)
{
    delete plan;
    return ok();
}

fma_status_t fma_workspace_size(fma_plan_t p, size_t *bytes)
{
    if (!p || !bytes) return fail(FMA_ERR_NULL, "fma_workspace_size: NULL argument");
    *bytes = p->ws_bytes;
    return ok();
}

fma_status_t fma_weights_len(fma_plan_t p, int64_t *floats)
{
    if (!p || !floats) return fail(FMA_ERR_NULL, "fma_weights_len: NULL argument");
    *floats = p->wlen;
    return ok();
}

fma_status_t fma_coarse_rows(fma_plan_t p, int64_t *rows)
{
    if (!p || !rows) return fail(FMA_ERR_NULL, "fma_coarse_rows: NULL argument");
    *rows = p->R;
    return ok();
}

fma_status_t fma_num_levels(fma_plan_t p, int32_t *levels)
{
    if (!p || !levels) return fail(FMA_ERR_NULL, "fma_num_levels: NULL argument");
    *levels = p->L;
    return ok();
}

}  // extern "C"

namespace {

size_t tensor_bytes(const fma_plan_s *p) { return (size_t)p->nslice * p->n * p->d * p->esize; }

bool empty_problem(const fma_plan_s *p) { return p->nslice == 0 || p->n == 0; }

fma_status_t check_tensor(const char *fn, const char *name, const void *x)
{
    if (!x) return fail(FMA_ERR_NULL, "%s: %s is NULL", fn, name);
    if (!aligned(x, 16)) return fail(FMA_ERR_ALIGN, "%s: %s is not 16-byte aligned", fn, name);
    return FMA_OK;
}

fma_status_t check_weights(const fma_plan_s *p, const char *fn, const float *wk, const float *wv)
{
    if (p->lv.nlev == 0) return FMA_OK;
    if (!wk || !wv) return fail(FMA_ERR_NULL, "%s: weights are NULL", fn);
    if (!aligned(wk, 4) || !aligned(wv, 4)) return fail(FMA_ERR_ALIGN, "%s: weights not 4-byte aligned", fn);
    return FMA_OK;
}

fma_status_t check_workspace(const fma_plan_s *p, const char *fn, const void *ws, size_t ws_bytes)
{
    if (p->lv.nlev == 0) return FMA_OK;
    if (!ws) return fail(FMA_ERR_WORKSPACE, "%s: workspace is NULL (need %zu bytes)", fn, p->ws_bytes);
    if (ws_bytes < p->ws_bytes)
        return fail(FMA_ERR_WORKSPACE, "%s: workspace of %zu bytes, need %zu", fn, ws_bytes, p->ws_bytes);
    if (!aligned(ws, 16)) return fail(FMA_ERR_ALIGN, "%s: workspace is not 16-byte aligned", fn);
    return FMA_OK;
}

fma_dev::CoarsenArgs coarsen_args(const fma_plan_s *p, const void *k, const void *v, const float *wk,
                                  const float *wv, void *ws)
{
    fma_dev::CoarsenArgs a;
    memset(&a, 0, sizeof(a));
    a.k = k;
    a.v = v;
    a.wk = wk;
    a.wv = wv;
    a.coarse = ws;
    a.part = reinterpret_cast<float *>(static_cast<char *>(ws) + p->part_offset);
    a.n = p->n;
    a.side = p->W;
    a.height = p->H;
    a.r = p->r;
    a.head_dim = p->d;
    a.two_d = p->desc.ndim == 2;
    a.nslice = p->nslice;
    a.heads = p->desc.heads > 0 ? p->desc.heads : 1;
    a.w_stride = p->desc.weights_per_head ? p->wlen : 0;
    a.R = (int)p->R;
    a.chunk = p->chunk;
    a.run = p->run;
    a.nchunk = p->nchunk;
    a.tiles_x = p->tiles_x;
    a.tiles_y = p->tiles_y;
    a.first_partial = p->first_partial;
    a.npartial = p->npartial;
    a.depth = p->depth;
    a.wave_lds = p->wave_lds;
    a.part_span = p->part_span;
    a.part_count = p->part_count;
    a.lv = p->lv;
    return a;
}

fma_dev::AttnArgs attend_args(const fma_plan_s *p, const void *q, const void *k, const void *v,
                              const void *ws, void *out)
{
    fma_dev::AttnArgs a;
    memset(&a, 0, sizeof(a));
    a.q = q;
    a.k = k;
    a.v = v;
    const size_t half = (size_t)p->nslice * p->R * p->d * p->esize;
    a.kbar = ws;
    a.vbar = ws ? static_cast<const char *>(ws) + half : nullptr;
    a.out = out;
    a.n = p->n;
    a.side = p->W;
    a.r = p->r;
    a.head_dim = p->d;
    a.nbx = p->nbx;
    a.nby = p->nby;
    a.qtile = p->desc.ndim == 1 ? p->r : p->r * p->r;
    a.tiles_per_slice = p->nblocks;
    a.nslice = p->nslice;
    a.R = (int)p->R;
    a.causal = p->desc.causal;
    a.nslot = p->nslot;
    a.slot_group = p->slot_group;
    a.rank = p->rank;
    a.norm_level = p->norm_level;
    a.ncoarse_tiles = (a.nslot + 63) / 64;
    a.scale_log2 = p->scale * 1.4426950408889634f;
    a.lv = p->lv;
    return a;
}

fma_status_t hip_status(const char *fn, hipError_t e)
{
    if (e != hipSuccess) return fail(FMA_ERR_HIP, "%s: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
    return ok();
}

fma_status_t do_coarsen(const fma_plan_s *p, const char *fn, const void *k, const void *v, const float *wk,
                        const float *wv, void *ws, size_t ws_bytes, void *stream)
{
    if (empty_problem(p)) return ok();   // nothing to read or write; pointers may be NULL
    fma_status_t st;
    if ((st = check_tensor(fn, "k", k)) || (st = check_tensor(fn, "v", v))) return st;
    if ((st = check_weights(p, fn, wk, wv))) return st;
    if ((st = check_workspace(p, fn, ws, ws_bytes))) return st;
    const size_t tb = tensor_bytes(p);
    if (p->lv.nlev > 0 && (overlap(ws, p->ws_bytes, k, tb) || overlap(ws, p->ws_bytes, v, tb)))
        return fail(FMA_ERR_ARG, "%s: workspace overlaps k or v", fn);
    if (empty_problem(p) || p->lv.nlev == 0) return ok();
    (void)hipGetLastError();
    const fma_dev::CoarsenArgs a = coarsen_args(p, k, v, wk, wv, ws);
    return hip_status(fn, fma_dev::launch_coarsen(a, p->desc.dtype == FMA_BF16, p->coarsen_smem,
                                                   static_cast<hipStream_t>(stream)));
}

fma_status_t do_attend(const fma_plan_s *p, const char *fn, const void *q, const void *k, const void *v,
                       const void *ws, size_t ws_bytes, void *out, void *stream)
{
    if (empty_problem(p)) return ok();
    fma_status_t st;
    if ((st = check_tensor(fn, "q", q)) || (st = check_tensor(fn, "k", k)) || (st = check_tensor(fn, "v", v)) ||
        (st = check_tensor(fn, "out", out)))
        return st;
    if ((st = check_workspace(p, fn, ws, ws_bytes))) return st;
    const size_t tb = tensor_bytes(p);
    if (overlap(out, tb, q, tb) || overlap(out, tb, k, tb) || overlap(out, tb, v, tb))
        return fail(FMA_ERR_ARG, "%s: out overlaps an input", fn);
    if (p->lv.nlev > 0 && overlap(out, tb, ws, p->ws_bytes)) return fail(FMA_ERR_ARG, "%s: out overlaps the workspace", fn);
    if (empty_problem(p)) return ok();
    (void)hipGetLastError();
    const fma_dev::AttnArgs a = attend_args(p, q, k, v, ws, out);
    const int geom = p->desc.ndim == 1 ? fma_dev::GEOM_1D : fma_dev::GEOM_2D;
    const bool bf16 = p->desc.dtype == FMA_BF16;
    // bf16 on the matrix-core tile-stream kernel; fp32 and blocks smaller
    // than a wave on the register-staged kernel
    if (bf16 && !p->generic)
        return hip_status(fn, fma_dev::launch_attend_bf16(a, geom, static_cast<hipStream_t>(stream)));
    return hip_status(fn, fma_dev::launch_attend(a, bf16, geom, static_cast<hipStream_t>(stream)));
}

// Argument checks of a forward call that do not involve the workspace.
fma_status_t check_forward_args(const fma_plan_s *p, const char *fn, const void *q, const void *k, const void *v,
                                const float *wk, const float *wv, const void *out)
{
    fma_status_t st;
    if ((st = check_tensor(fn, "q", q)) || (st = check_tensor(fn, "out", out))) return st;
    if ((st = check_tensor(fn, "k", k)) || (st = check_tensor(fn, "v", v))) return st;
    if ((st = check_weights(p, fn, wk, wv))) return st;
    const size_t tb = tensor_bytes(p);
    if (overlap(out, tb, q, tb) || overlap(out, tb, k, tb) || overlap(out, tb, v, tb))
        return fail(FMA_ERR_ARG, "%s: out overlaps an input", fn);
    return FMA_OK;
}

fma_status_t do_forward(const fma_plan_s *p, int ndim, const char *fn, const void *q, const void *k, const void *v,
                        const float *wk, const float *wv, void *out, void *ws, size_t ws_bytes, void *stream)
{
    if (!p) return fail(FMA_ERR_NULL, "%s: plan is NULL", fn);
    if (p->desc.ndim != ndim) return fail(FMA_ERR_SHAPE, "%s: plan is %dD", fn, p->desc.ndim);
    if (p->linear) return fail(FMA_ERR_ARG, "%s: the plan is FMA-linear, use fma_forward_linear", fn);
    if (empty_problem(p)) return ok();
    fma_status_t st;
    // validate the attention stage too before anything is launched
    if ((st = check_forward_args(p, fn, q, k, v, wk, wv, out))) return st;
    const size_t tb = tensor_bytes(p);
    if (p->lv.nlev > 0 && ws && overlap(ws, p->ws_bytes, q, tb)) return fail(FMA_ERR_ARG, "%s: workspace overlaps q", fn);
    if ((st = check_workspace(p, fn, ws, ws_bytes))) return st;
    if (p->lv.nlev > 0 && overlap(out, tb, ws, p->ws_bytes)) return fail(FMA_ERR_ARG, "%s: out overlaps the workspace", fn);
    if ((st = do_coarsen(p, fn, k, v, wk, wv, ws, ws_bytes, stream))) return st;
    return do_attend(p, fn, q, k, v, ws, ws_bytes, out, stream);
}

}  // namespace

extern "C" {

fma_status_t fma_forward_1d(fma_plan_t plan, const void *q, const void *k, const void *v, const float *wk,
                            const float *wv, void *out, void *workspace, size_t workspace_bytes, void *stream)
{
    return do_forward(plan, 1, "fma_forward_1d", q, k, v, wk, wv, out, workspace, workspace_bytes, stream);
}

fma_status_t fma_forward_2d(fma_plan_t plan, const void *q, const void *k, const void *v, const float *wk,
                            const float *wv, void *out, void *workspace, size_t workspace_bytes, void *stream)
{
    return do_forward(plan, 2, "fma_forward_2d", q, k, v, wk, wv, out, workspace, workspace_bytes, stream);
}

fma_status_t fma_coarsen(fma_plan_t plan, const void *k, const void *v, const float *wk, const float *wv,
                         void *workspace, size_t workspace_bytes, void *stream)
{
    if (!plan) return fail(FMA_ERR_NULL, "fma_coarsen: plan is NULL");
    return do_coarsen(plan, "fma_coarsen", k, v, wk, wv, workspace, workspace_bytes, stream);
}

fma_status_t fma_attend(fma_plan_t plan, const void *q, const void *k, const void *v, const void *workspace,
                        size_t workspace_bytes, void *out, void *stream)
{
    if (!plan) return fail(FMA_ERR_NULL, "fma_attend: plan is NULL");
    if (plan->linear) return fail(FMA_ERR_ARG, "fma_attend: the plan is FMA-linear, use fma_forward_linear");
    return do_attend(plan, "fma_attend", q, k, v, workspace, workspace_bytes, out, stream);
}

fma_status_t fma_interaction_lists(fma_plan_t p, int32_t *dev_out, void *stream)
{
    if (!p) return fail(FMA_ERR_NULL, "fma_interaction_lists: plan is NULL");
    if (!dev_out) return fail(FMA_ERR_NULL, "fma_interaction_lists: dev_out is NULL");
    if (!aligned(dev_out, 4)) return fail(FMA_ERR_ALIGN, "fma_interaction_lists: dev_out not 4-byte aligned");
    if (p->lv.nlev == 0) return ok();
    (void)hipGetLastError();
    return hip_status("fma_interaction_lists",
                      fma_dev::launch_lists(p->desc.ndim == 2, p->nblocks, p->nby, p->desc.causal, p->rlv, dev_out,
                                            static_cast<hipStream_t>(stream)));
}

fma_status_t fma_forward_linear(fma_plan_t p, const void *q, const void *k, const void *v, const float *wq,
                                const float *wk, const float *wv, void *out, void *workspace, size_t workspace_bytes,
                                void *stream)
{
    const char *fn = "fma_forward_linear";
    if (!p) return fail(FMA_ERR_NULL, "%s: plan is NULL", fn);
    if (!p->linear) return fail(FMA_ERR_ARG, "%s: the plan does not downsample queries (query_downsample = 0)", fn);
    if (empty_problem(p)) return ok();
    fma_status_t st;
    if ((st = check_tensor(fn, "q", q)) || (st = check_tensor(fn, "k", k)) || (st = check_tensor(fn, "v", v)) ||
        (st = check_tensor(fn, "out", out)))
        return st;
    if ((st = check_weights(p, fn, wk, wv))) return st;
    if (p->lv.nlev > 0) {
        if (!wq) return fail(FMA_ERR_NULL, "%s: wq is NULL", fn);
        if (!aligned(wq, 4)) return fail(FMA_ERR_ALIGN, "%s: wq not 4-byte aligned", fn);
    }
    if ((st = check_workspace(p, fn, workspace, workspace_bytes))) return st;
    const size_t tb = tensor_bytes(p);
    if (overlap(out, tb, q, tb) || overlap(out, tb, k, tb) || overlap(out, tb, v, tb))
        return fail(FMA_ERR_ARG, "%s: out overlaps an input", fn);
    if (p->lv.nlev > 0 && (overlap(out, tb, workspace, p->ws_bytes) || overlap(workspace, p->ws_bytes, q, tb) ||
                           overlap(workspace, p->ws_bytes, k, tb) || overlap(workspace, p->ws_bytes, v, tb)))
        return fail(FMA_ERR_ARG, "%s: the workspace overlaps a tensor", fn);
    (void)hipGetLastError();
    hipStream_t hs = static_cast<hipStream_t>(stream);
    char *ws = static_cast<char *>(workspace);
    if (p->lv.nlev > 0) {
        // K_bar, V_bar; then the coarse queries (the same coarsening on Q twice:
        // its first half is Q_bar, the second an unused copy)
        hipError_t e = fma_dev::launch_coarsen(coarsen_args(p, k, v, wk, wv, ws), p->desc.dtype == FMA_BF16,
                                               p->coarsen_smem, hs);
        if (e != hipSuccess) return hip_status(fn, e);
        // Q_bar: with an even number of slices whose second half starts on a
        // head boundary (or shared weights) the two halves of Q take the places
        // of the two tensors, so one pass covers Q and writes Q_bar as
        // [S][R][d]; otherwise Q is coarsened twice (the second copy unused)
        fma_dev::CoarsenArgs cq = coarsen_args(p, q, q, wq, wq, ws + p->lin_q_offset);
        const int heads = p->desc.heads > 0 ? p->desc.heads : 1;
        if (p->nslice % 2 == 0 && (!p->desc.weights_per_head || (p->nslice / 2) % heads == 0)) {
            cq.v = static_cast<const char *>(q) + tensor_bytes(p) / 2;
            cq.nslice = p->nslice / 2;
        }
        e = fma_dev::launch_coarsen(cq, p->desc.dtype == FMA_BF16, p->coarsen_smem, hs);
        if (e != hipSuccess) return hip_status(fn, e);
    }
    fma_dev::AttnArgs a = attend_args(p, q, k, v, ws, out);
    a.qbar = p->lv.nlev > 0 ? ws + p->lin_q_offset : nullptr;
    const int geom = p->desc.ndim == 1 ? fma_dev::GEOM_1D : fma_dev::GEOM_2D;
    // bf16: every block's far field (M, Z, U) first, then the fused
    // matrix-core kernel; fp32 and blocks smaller than a wave: the
    // register-staged kernel does both
    if (p->desc.dtype == FMA_BF16 && !p->generic) {
        if (p->lv.nlev > 0) {
            a.lin_far = reinterpret_cast<float *>(ws + p->lin_far_offset);
            a.lin_far_elems = (long long)p->nslice * p->nblocks * (p->d + 2);
            const hipError_t e = fma_dev::launch_lin_far(a, geom, hs);
            if (e != hipSuccess) return hip_status(fn, e);
        }
        return hip_status(fn, fma_dev::launch_attend_bf16(a, geom, hs));
    }
    return hip_status(fn, fma_dev::launch_attend(a, p->desc.dtype == FMA_BF16, geom, hs));
}

fma_status_t fma_backward_workspace_size(fma_plan_t p, size_t *bytes)
{
    if (!p || !bytes) return fail(FMA_ERR_NULL, "fma_backward_workspace_size: NULL argument");
    *bytes = p->bw_bytes;
    return ok();
}

}  // extern "C"

namespace {

// Both backward entry points: FMA (wq = dwq = NULL) and FMA-linear.
fma_status_t backward_impl(const char *fn, fma_plan_t p, const void *q, const void *k, const void *v,
                           const float *wk, const float *wv, const float *wq, const void *out, const void *dout,
                           void *dq, void *dk, void *dv, float *dwk, float *dwv, float *dwq, void *workspace,
                           size_t workspace_bytes, void *stream)
{
    if (!p) return fail(FMA_ERR_NULL, "%s: plan is NULL", fn);
    if (p->d != fma_dev::kHeadDim)
        return fail(FMA_ERR_UNSUPPORTED, "%s: the backward is built for head_dim 64 (plan: %d)", fn, p->d);
    // the FMA-linear dq kernel indexes tokens and its 32-token workgroups in 32 bits
    if (p->linear && (p->n > 0x7fffffffLL - 32 || (long long)p->nslice * ((p->n + 31) / 32) > 0x7fffffffLL))
        return fail(FMA_ERR_SHAPE, "%s: FMA-linear backward needs seq_len < 2^31 - 32 and B*H*seq_len/32 < 2^31", fn);
    if (empty_problem(p)) return ok();
    fma_status_t st;
    const void *ins[5] = {q, k, v, out, dout};
    const char *in_names[5] = {"q", "k", "v", "out", "dout"};
    void *outs[3] = {dq, dk, dv};
    const char *out_names[3] = {"dq", "dk", "dv"};
    for (int i = 0; i < 5; ++i)
        if ((st = check_tensor(fn, in_names[i], ins[i]))) return st;
    for (int i = 0; i < 3; ++i)
        if ((st = check_tensor(fn, out_names[i], outs[i]))) return st;
    const int nlev = p->lv.nlev;
    if (nlev > 0) {
        if ((st = check_weights(p, fn, wk, wv))) return st;
        if (!dwk || !dwv) return fail(FMA_ERR_NULL, "%s: weight gradients are NULL", fn);
        if (!aligned(dwk, 4) || !aligned(dwv, 4)) return fail(FMA_ERR_ALIGN, "%s: weight gradients not 4-byte aligned", fn);
        if (p->linear) {
            if (!wq || !dwq) return fail(FMA_ERR_NULL, "%s: query weights or their gradient are NULL", fn);
            if (!aligned(wq, 4) || !aligned(dwq, 4))
                return fail(FMA_ERR_ALIGN, "%s: query weights or their gradient not 4-byte aligned", fn);
        }
    }
    if (!workspace) return fail(FMA_ERR_WORKSPACE, "%s: workspace is NULL (need %zu bytes)", fn, p->bw_bytes);
    if (workspace_bytes < p->bw_bytes)
        return fail(FMA_ERR_WORKSPACE, "%s: workspace of %zu bytes, need %zu", fn, workspace_bytes, p->bw_bytes);
    if (!aligned(workspace, 16)) return fail(FMA_ERR_ALIGN, "%s: workspace is not 16-byte aligned", fn);
    const size_t tb = tensor_bytes(p);
    const int heads_w = p->desc.weights_per_head ? (p->desc.heads > 0 ? p->desc.heads : 1) : 1;
    const size_t wb = (size_t)heads_w * p->wlen * sizeof(float);
    // outputs overlap no input, no other output and not the workspace
    for (int i = 0; i < 3; ++i) {
        for (int j = 0; j < 5; ++j)
            if (overlap(outs[i], tb, ins[j], tb)) return fail(FMA_ERR_ARG, "%s: %s overlaps %s", fn, out_names[i], in_names[j]);
        for (int j = i + 1; j < 3; ++j)
            if (overlap(outs[i], tb, outs[j], tb)) return fail(FMA_ERR_ARG, "%s: %s overlaps %s", fn, out_names[i], out_names[j]);
        if (overlap(outs[i], tb, workspace, p->bw_bytes)) return fail(FMA_ERR_ARG, "%s: %s overlaps the workspace", fn, out_names[i]);
    }
    for (int j = 0; j < 5; ++j)
        if (overlap(workspace, p->bw_bytes, ins[j], tb)) return fail(FMA_ERR_ARG, "%s: workspace overlaps %s", fn, in_names[j]);
    if (nlev > 0) {
        const void *wouts[2] = {dwk, dwv};
        for (int i = 0; i < 2; ++i) {
            if (overlap(wouts[i], wb, workspace, p->bw_bytes) || overlap(wouts[i], wb, wk, wb) ||
                overlap(wouts[i], wb, wv, wb))
                return fail(FMA_ERR_ARG, "%s: a weight gradient overlaps the workspace or the weights", fn);
            for (int j = 0; j < 5; ++j)
                if (overlap(wouts[i], wb, ins[j], tb)) return fail(FMA_ERR_ARG, "%s: a weight gradient overlaps an input", fn);
            for (int j = 0; j < 3; ++j)
                if (overlap(wouts[i], wb, outs[j], tb)) return fail(FMA_ERR_ARG, "%s: a weight gradient overlaps an output", fn);
        }
        if (overlap(dwk, wb, dwv, wb)) return fail(FMA_ERR_ARG, "%s: dwk overlaps dwv", fn);
        if (p->linear) {
            if (overlap(dwq, wb, workspace, p->bw_bytes) || overlap(dwq, wb, wk, wb) || overlap(dwq, wb, wv, wb) ||
                overlap(dwq, wb, wq, wb) || overlap(dwq, wb, dwk, wb) || overlap(dwq, wb, dwv, wb) ||
                overlap(dwk, wb, wq, wb) || overlap(dwv, wb, wq, wb))
                return fail(FMA_ERR_ARG, "%s: dwq overlaps the workspace, the weights or another gradient", fn);
            for (int j = 0; j < 5; ++j)
                if (overlap(dwq, wb, ins[j], tb)) return fail(FMA_ERR_ARG, "%s: dwq overlaps an input", fn);
            for (int j = 0; j < 3; ++j)
                if (overlap(dwq, wb, outs[j], tb)) return fail(FMA_ERR_ARG, "%s: dwq overlaps an output", fn);
        }
    }
    (void)hipGetLastError();
    hipStream_t hs = static_cast<hipStream_t>(stream);
    char *const wsb = static_cast<char *>(workspace);
    if (nlev > 0) {
        const fma_dev::CoarsenArgs ca = coarsen_args(p, k, v, wk, wv, workspace);
        hipError_t e = fma_dev::launch_coarsen(ca, p->desc.dtype == FMA_BF16, p->coarsen_smem, hs);
        if (e != hipSuccess) return hip_status(fn, e);
        if (p->linear) {
            // the coarse queries, as the linear forward forms them
            fma_dev::CoarsenArgs cq = coarsen_args(p, q, q, wq, wq, wsb + p->lin_q_offset);
            const int heads = p->desc.heads > 0 ? p->desc.heads : 1;
            if (p->nslice % 2 == 0 && (!p->desc.weights_per_head || (p->nslice / 2) % heads == 0)) {
                cq.v = static_cast<const char *>(q) + tensor_bytes(p) / 2;
                cq.nslice = p->nslice / 2;
            }
            e = fma_dev::launch_coarsen(cq, p->desc.dtype == FMA_BF16, p->coarsen_smem, hs);
            if (e != hipSuccess) return hip_status(fn, e);
        }
    }
    fma_dev::BwdArgs a;
    memset(&a, 0, sizeof(a));
    char *ws = static_cast<char *>(workspace);
    const size_t half = (size_t)p->nslice * p->R * p->d * p->esize;
    a.q = q;
    a.k = k;
    a.v = v;
    a.out = out;
    a.dout = dout;
    a.kbar = ws;
    a.vbar = ws + half;
    a.wk = wk;
    a.wv = wv;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.dwk = dwk;
    a.dwv = dwv;
    a.lse = reinterpret_cast<float *>(ws + p->bw_lse);
    a.delta = reinterpret_cast<float *>(ws + p->bw_delta);
    a.part = reinterpret_cast<float *>(ws + p->bw_part);
    const size_t cb = (size_t)p->nslice * p->R * fma_dev::kHeadDim;
    a.dkbar = reinterpret_cast<float *>(ws + p->bw_cbar);
    a.dvbar = a.dkbar + cb;
    const size_t sn = (size_t)p->nslice * p->n;
    a.dotk = reinterpret_cast<float *>(ws + p->bw_dot);
    a.dotv = a.dotk + sn * nlev;
    a.n = p->n;
    a.side = p->W;
    a.height = p->H;
    a.r = p->r;
    a.nbx = p->nbx;
    a.nby = p->nby;
    a.qtile = p->desc.ndim == 1 ? p->r : p->r * p->r;
    a.nblocks = p->nblocks;
    a.npart = 0;   // set per launch shape by the backward launcher
    a.nslice = p->nslice;
    a.heads = p->desc.heads > 0 ? p->desc.heads : 1;
    a.heads_w = heads_w;
    a.R = (int)p->R;
    a.causal = p->desc.causal;
    a.nslot = p->nslot;
    a.rank = p->rank;
    a.norm_level = p->norm_level;
    a.slot_group = p->slot_group;
    a.w_stride = p->desc.weights_per_head ? p->wlen : 0;
    a.wlen = (int)p->wlen;
    a.scale = p->scale;
    a.scale_log2 = p->scale * 1.4426950408889634f;
    a.io_elems = (long long)sn * fma_dev::kHeadDim;
    a.coarse_elems = (long long)cb;
    a.part_elems = (long long)p->bw_part_floats;
    a.slice0 = 0;
    a.pslices = p->bw_pslices;
    a.dot_elems = (long long)sn * nlev;
    a.lse_elems = (long long)sn;
    a.w_elems = (long long)heads_w * p->wlen;
    a.lv = p->lv;
    if (p->linear) {
        a.qbar = nlev > 0 ? wsb + p->lin_q_offset : nullptr;
        a.wq = wq;
        a.dwq = dwq;
        a.qpart = reinterpret_cast<float *>(ws + p->bw_qpart);
        a.dqbar = reinterpret_cast<float *>(ws + p->bw_dqbar);
        a.dqn = reinterpret_cast<float *>(ws + p->bw_dqn);
        a.dotq = reinterpret_cast<float *>(ws + p->bw_dotq);
        a.qpart_elems = (long long)p->nslice * p->npart_max * nlev * fma_dev::kHeadDim;
        a.dqn_elems = (long long)sn * fma_dev::kHeadDim;
        if (nlev == 0) a.qbar = wsb + p->lin_q_offset;   // selects the linear kernels; never read
    }
    return hip_status(fn, fma_dev::launch_backward(a, p->desc.dtype == FMA_BF16, p->desc.ndim == 2, hs));
}

}  // namespace

extern "C" {

fma_status_t fma_backward(fma_plan_t p, const void *q, const void *k, const void *v, const float *wk, const float *wv,
                          const void *out, const void *dout, void *dq, void *dk, void *dv, float *dwk, float *dwv,
                          void *workspace, size_t workspace_bytes, void *stream)
{
    const char *fn = "fma_backward";
    if (p && p->linear)
        return fail(FMA_ERR_ARG, "%s: plan is FMA-linear; use fma_backward_linear", fn);
    return backward_impl(fn, p, q, k, v, wk, wv, nullptr, out, dout, dq, dk, dv, dwk, dwv, nullptr, workspace,
                         workspace_bytes, stream);
}

fma_status_t fma_backward_linear(fma_plan_t p, const void *q, const void *k, const void *v, const float *wk,
                                 const float *wv, const float *wq, const void *out, const void *dout, void *dq,
                                 void *dk, void *dv, float *dwk, float *dwv, float *dwq, void *workspace,
                                 size_t workspace_bytes, void *stream)
{
    const char *fn = "fma_backward_linear";
    if (p && !p->linear) return fail(FMA_ERR_ARG, "%s: plan is not FMA-linear; use fma_backward", fn);
    return backward_impl(fn, p, q, k, v, wk, wv, wq, out, dout, dq, dk, dv, dwk, dwv, dwq, workspace,
                         workspace_bytes, stream);
}

fma_status_t fma_dense_reference(fma_plan_t p, const void *q, const void *k, const void *v, void *out, void *stream)
{
    const char *fn = "fma_dense_reference";
    if (!p) return fail(FMA_ERR_NULL, "%s: plan is NULL", fn);
    if (empty_problem(p)) return ok();
    fma_status_t st;
    if ((st = check_tensor(fn, "q", q)) || (st = check_tensor(fn, "k", k)) || (st = check_tensor(fn, "v", v)) ||
        (st = check_tensor(fn, "out", out)))
        return st;
    const size_t tb = tensor_bytes(p);
    if (overlap(out, tb, q, tb) || overlap(out, tb, k, tb) || overlap(out, tb, v, tb))
        return fail(FMA_ERR_ARG, "%s: out overlaps an input", fn);
    if (p->n % 64) return fail(FMA_ERR_UNSUPPORTED, "%s: seq_len must be a multiple of 64", fn);
    if (empty_problem(p)) return ok();
    fma_dev::AttnArgs a = attend_args(p, q, k, v, nullptr, out);
    a.qtile = p->n % 128 == 0 ? 128 : 64;
    a.tiles_per_slice = (int)(p->n / a.qtile);
    a.ncoarse_tiles = 0;
    a.nslot = 0;
    a.norm_level = 0;
    a.lv.nlev = 0;
    (void)hipGetLastError();
    if (p->desc.dtype == FMA_BF16 && p->d == fma_dev::kHeadDim)
        return hip_status(fn, fma_dev::launch_attend_bf16(a, fma_dev::GEOM_DENSE, static_cast<hipStream_t>(stream)));
    return hip_status(fn, fma_dev::launch_attend(a, p->desc.dtype == FMA_BF16, fma_dev::GEOM_DENSE,
                                                 static_cast<hipStream_t>(stream)));
}

}  // extern "C"

extern "C" fma_status_t fma_plan_params(fma_plan_t p, int64_t *out, int32_t capacity, int32_t *count)
{
    const char *fn = "fma_plan_params";
    if (!p || !out || !count) return fail(FMA_ERR_NULL, "%s: NULL argument", fn);
    const int nsets = p->lv.nlev;
    const int need = 41 + 6 * nsets;
    *count = need;
    if (capacity < need) return fail(FMA_ERR_WORKSPACE, "%s: capacity %d, need %d", fn, capacity, need);
    const int heads = p->desc.heads > 0 ? p->desc.heads : 1;
    const int64_t v[36] = {
        p->n, p->W, p->r, p->nbx, p->desc.ndim == 1 ? p->r : (int64_t)p->r * p->r, p->nblocks, p->nslice, p->R,
        p->desc.causal, p->nslot, p->slot_group, p->rank, p->norm_level, p->desc.ndim, p->esize, heads,
        p->desc.weights_per_head ? p->wlen : 0, p->wlen, nsets, p->chunk, p->run, p->nchunk, p->tiles_y,
        p->first_partial, p->npartial, p->part_span, p->part_count, p->depth, p->wave_lds, (int64_t)p->coarsen_smem,
        (int64_t)p->part_offset, (int64_t)p->coarse_bytes, (int64_t)p->ws_bytes, p->linear,
        p->desc.weights_per_head ? heads : 1, p->desc.dtype};
    for (int i = 0; i < 36; ++i) out[i] = v[i];
    out[36] = p->desc.ndim == 2 && !p->generic &&
              fma_dev::pair_cells_2d(p->r, p->nby, p->nslot, p->norm_level, p->linear, p->desc.dtype == FMA_BF16);
    out[37] = p->H;
    out[38] = p->nby;
    out[39] = p->tiles_x;
    out[40] = p->d;
    for (int e = 0; e < nsets; ++e) {
        out[41 + 6 * e + 0] = p->lv.off[e];
        out[41 + 6 * e + 1] = p->lv.M[e];
        out[41 + 6 * e + 2] = p->lv.My[e];
        out[41 + 6 * e + 3] = p->lv.size[e];
        out[41 + 6 * e + 4] = p->lv.woff[e];
        out[41 + 6 * e + 5] = p->lv.lvl[e];
    }
    return ok();
}

extern "C" fma_status_t fma_stream_reference(const void *src, size_t src_bytes, void *dst, size_t dst_bytes,
                                             int32_t write_every, void *stream)
{
    const char *fn = "fma_stream_reference";
    if (!src || !dst) return fail(FMA_ERR_NULL, "%s: src and dst must not be NULL", fn);
    if (!aligned(src, 16) || !aligned(dst, 16)) return fail(FMA_ERR_ALIGN, "%s: buffers must be 16-byte aligned", fn);
    if (src_bytes % 16) return fail(FMA_ERR_SHAPE, "%s: src_bytes must be a multiple of 16", fn);
    if (write_every != 1 && write_every != 2 && write_every != 4 && write_every != 8 && write_every != 16 &&
        write_every != 32 && write_every != 64 && write_every != 128 && write_every != 256)
        return fail(FMA_ERR_ARG, "%s: write_every must be a power of two from 1 to 256, got %d", fn, write_every);
    const long long nwords = (long long)(src_bytes / 16);
    const long long need = fma_dev::stream_ref_dst_words(nwords, write_every);
    if (dst_bytes < (size_t)need * 16)
        return fail(FMA_ERR_WORKSPACE, "%s: dst of %zu bytes, need %lld", fn, dst_bytes, need * 16);
    if (overlap(src, src_bytes, dst, dst_bytes)) return fail(FMA_ERR_ARG, "%s: src overlaps dst", fn);
    (void)hipGetLastError();
    return hip_status(fn, fma_dev::launch_stream_ref(src, nwords, dst, need, write_every,
                                                     static_cast<hipStream_t>(stream)));
}

// ------------------------------------------------------------------------
// Allocation-free forward (fma_forward_static): the workspace of the forward
// pass -- coarse keys and values, fp32 partial sums of the wide coarse sets
// -- lives in a file-scope device array instead of a caller's buffer.  Each
// GPU holds its own copy of the array (for the life of the process); its
// device address is looked up once per device and kept.  The array's name
// in host code is only a host-side stand-in: every launch takes the looked-up
// address.
namespace {

constexpr size_t kStaticScratchBytes = (size_t)32 << 20;   // 32 MiB per GPU
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

std::once_flag g_scratch_once[kMaxDevices];
hipError_t g_scratch_status[kMaxDevices];
void *g_scratch_ptr[kMaxDevices];

// Device address of `scratch` on the current device (looked up on the first
// call per device, with that device current).
fma_status_t static_scratch(const char *fn, void **ptr)
{
    int dev = -1;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(fn, e);
    if (dev < 0 || dev >= kMaxDevices) return fail(FMA_ERR_HIP, "%s: device %d out of range", fn, dev);
    std::call_once(g_scratch_once[dev], [dev]() {
        void *p = nullptr;
        g_scratch_status[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch_ptr[dev] = g_scratch_status[dev] == hipSuccess ? p : nullptr;
    });
    if (g_scratch_status[dev] != hipSuccess)
        return fail(FMA_ERR_HIP, "%s: device address of the static scratch buffer: HIP error %d (%s)", fn,
                    (int)g_scratch_status[dev], hipGetErrorString(g_scratch_status[dev]));
    if (!g_scratch_ptr[dev] || !aligned(g_scratch_ptr[dev], 256))
        return fail(FMA_ERR_HIP, "%s: the static scratch buffer has no usable device address", fn);
    *ptr = g_scratch_ptr[dev];
    return FMA_OK;
}

}  // namespace

extern "C" {

fma_status_t fma_forward_static(fma_plan_t p, const void *q, const void *k, const void *v, const float *wk,
                                const float *wv, void *out, void *stream)
{
    const char *fn = "fma_forward_static";
    if (!p) return fail(FMA_ERR_NULL, "%s: plan is NULL", fn);
    if (p->linear) return fail(FMA_ERR_ARG, "%s: the plan is FMA-linear, use fma_forward_linear", fn);
    if (p->ws_bytes > kStaticScratchBytes)
        return fail(FMA_ERR_WORKSPACE,
                    "%s: the plan needs %zu bytes of workspace, the static scratch buffer holds %zu; use "
                    "fma_forward_%dd with a caller workspace", fn, p->ws_bytes, kStaticScratchBytes, p->desc.ndim);
    if (empty_problem(p)) return ok();
    // every argument is checked before the device is touched
    fma_status_t st = check_forward_args(p, fn, q, k, v, wk, wv, out);
    if (st != FMA_OK) return st;
    void *ws = nullptr;
    if (p->lv.nlev > 0 && (st = static_scratch(fn, &ws)) != FMA_OK) return st;
    return do_forward(p, p->desc.ndim, fn, q, k, v, wk, wv, out, ws, p->lv.nlev > 0 ? kStaticScratchBytes : 0,
                      stream);
}

}  // extern "C"
