/*
 * fma_oracle.c -- CPU oracle for the Fast Multipole Attention (FMA) forward pass.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * reference that the GPU path is checked against.  Only the tests, the smoke
 * check and the benchmark's CPU-baseline leg may load it.  It shares no code,
 * header, table or constant with the HIP library and it includes nothing from
 * the product package.
 *
 * Everything is computed in double precision, directly from the definitions
 * of Section 3 ("Fast Multipole Attention") of Kang, Tran & De Sterck,
 * "Fast Multipole Attention: A Scalable Multilevel Attention Mechanism for
 * Text and Images" (arXiv 2310.11960):
 *
 *   - hierarchy depth L = ceil(log2(n/r))                  (Sec. 3, "FMA in 1D")
 *   - level-l groups of length r*2^(l-1), clipped to [n]   (Sec. 3, "FMA in 1D")
 *   - learned aggregation of keys / values inside a group  (Eq. agg1d)
 *   - near field N(i): base blocks at distance <= 1        (Sec. 3, "Near field")
 *   - far field F_l(i): level-l blocks at distance <= 1,
 *     minus everything already assigned                     (Sec. 3, "Far field")
 *   - the groups G_l(i) that lie inside F_l(i)             (Sec. 3, beta weights)
 *   - output = near-field weights times values + coarse
 *     weights times aggregated values                      (Eq. fma1d)
 *   - the 2D quadtree analogues                            (Sec. 3, "FMA in 2D",
 *                                                            Eq. agg2d, Eq. fma2d)
 *
 * Index sets are built by literally applying the set-builder definitions to
 * every token j of the sequence (brute force, O(n) per base block and level);
 * no closed form is used anywhere in this file.
 *
 * Readings taken where the paper is silent (documented with the design notes):
 *   - normalisation: by default ONE softmax over the union of near tokens and
 *     far groups (norm_mode 0).  norm_mode 1 applies the printed per-set
 *     normalisation (alpha over N(i), each beta^l over G_l(i)) literally.
 *   - causal use (the paper says FMA works autoregressively but defines no
 *     mask): a near token j is visible to query i iff j <= i; a far group is
 *     visible iff all of its tokens are <= i.
 *   - 2D token t = x*W + y with x the row index; pi^(x) runs along rows.
 *   - a group / square that is clipped by the sequence end (n/r not a power
 *     of two) aggregates only its existing tokens, with weights indexed by
 *     the offset from the group start.
 *   - coarse level rank p (Sec. 3, "Coarse level rank p"): every level learns
 *     p basis vectors, every group stores p aggregated keys and values, and
 *     the query scores each of the p representatives as its own source (each
 *     with its own value), normalised with the other sources as above.
 *     Layouts: the weights of level l hold basis s at offset
 *     p*r*(2^(l-1)-1) + s*s_l (2D: p*2r*(2^(l-1)-1) + s*2*s_l, [pi_x | pi_y]
 *     per basis); coarse row of level l, basis s, group m =
 *     p*(rows of the levels below l) + s*M_l + m (2D: M_l^2 squares per
 *     basis).  p = 1 is the default single-vector form.
 *
 * FMA-linear (query downsampling, Sec. 3 remark after Eq. fma1d / Eq. fma2d;
 * the paper gives no formula, this is the reading used here): the queries
 * of every level-l group are aggregated with learned weights pi^q (laid out
 * like pi^k, rank 1) into a coarse query, and every token of the group scores
 * its level-l far-field groups with that coarse query instead of its own; the
 * near field keeps the fine query; one softmax as above.  Causal use is
 * rejected: a group's coarse query mixes the queries of later tokens.
 *
 * Backward (gradients of a scalar loss with upstream dO, for training the
 * weights end to end, Sec. 1 / Sec. 3): the same per-row sources, the
 * softmax derivative dS_t = P_t (dO.v_t - D) with D = sum over the row's
 * (per-set: the set's) sources of P_t dO.v_t, dq = tau sum dS_t k_t,
 * dk_t += tau dS_t q, dv_t += P_t dO (k_t, v_t fine or coarse), then the
 * coarsening, which is linear in the tokens and in the weights:
 * dx_j += pi[j - start] dbar_G and dpi[o] += x_{start+o} . dbar_G.
 *
 * parity pinned by: dense-attention special case (n = r, n = 2r), per-row
 * brute-force sets, disjoint cover, closed-form work counts, row weights
 * summing to one, causality under perturbation, reversal / transpose
 * equivariance, an independent dense masked formulation over augmented keys,
 * coarsening special cases (one-hot and uniform weights), linearity in V.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define FMAO_OK 0
#define FMAO_ERR_ARG 1
#define FMAO_ERR_COVER 2
#define FMAO_ERR_ALLOC 3

/* ------------------------------------------------------------------ */
/* Geometry (Sec. 3): L = ceil(log2(ratio)), 0 when ratio <= 1.        */
/* ------------------------------------------------------------------ */
int fmao_num_levels(int64_t ratio)
{
    int L = 0;
    int64_t p = 1;
    while (p < ratio) {
        p *= 2;
        L += 1;
    }
    return L;
}

static int64_t iabs64(int64_t a) { return a < 0 ? -a : a; }
static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

/* group length at coarse level l >= 1: r * 2^(l-1) */
static int64_t group_len(int64_t r, int l) { return r << (l - 1); }

/* Number of coarse rows over all levels: sum_l M_l, M_l = ceil(len/s_l). */
int64_t fmao_coarse_rows_1d(int64_t n, int64_t r)
{
    if (r <= 0 || n <= 0 || n % r) return -1;
    int L = fmao_num_levels(n / r);
    int64_t R = 0;
    for (int l = 1; l < L; ++l) R += ceil_div(n, group_len(r, l));
    return R;
}

/* 2D maps of H rows and W columns (token t = x*W + y): the hierarchy runs
 * until the longer side has two groups, L = ceil(log2(max(H, W) / r)); a
 * level has ceil(H/s_l) x ceil(W/s_l) groups. */
static int levels_2d(int64_t H, int64_t W, int64_t r) { return fmao_num_levels((H > W ? H : W) / r); }

int64_t fmao_coarse_rows_2d_hw(int64_t H, int64_t W, int64_t r)
{
    if (r <= 0 || W <= 0 || H <= 0 || W % r || H % r) return -1;
    int L = levels_2d(H, W, r);
    int64_t R = 0;
    for (int l = 1; l < L; ++l) R += ceil_div(H, group_len(r, l)) * ceil_div(W, group_len(r, l));
    return R;
}

int64_t fmao_coarse_rows_2d(int64_t W, int64_t r) { return fmao_coarse_rows_2d_hw(W, W, r); }

/* ------------------------------------------------------------------ */
/* 1D index sets, by definition.                                        */
/*                                                                      */
/* label[j] = 0 if j in N(i), l if j in F_l(i).  For every level the    */
/* groups G_{l,m} contained in F_l(i) are listed in ascending m in      */
/* grp[l][*] (count ngrp[l]).  The sets depend on i only through        */
/* b0(i) = floor(i/r), because r*2^l is a multiple of r; the caller     */
/* passes any row i of the base block.                                   */
/* ------------------------------------------------------------------ */
typedef struct {
    int L;
    int8_t *label;       /* [n] */
    int64_t *grp;        /* [L][gcap] group indices m */
    int64_t *ngrp;       /* [L] */
    int64_t gcap;
} sets_t;

static int sets_alloc(sets_t *s, int64_t n, int L)
{
    s->L = L;
    s->gcap = n > 0 ? n : 1;
    s->label = (int8_t *)malloc((size_t)(n > 0 ? n : 1));
    s->grp = (int64_t *)malloc(sizeof(int64_t) * (size_t)(L > 0 ? L : 1) * (size_t)s->gcap);
    s->ngrp = (int64_t *)calloc((size_t)(L > 0 ? L : 1), sizeof(int64_t));
    return (s->label && s->grp && s->ngrp) ? FMAO_OK : FMAO_ERR_ALLOC;
}

static void sets_free(sets_t *s)
{
    free(s->label);
    free(s->grp);
    free(s->ngrp);
}

static int build_sets_1d(int64_t n, int64_t r, int64_t i, sets_t *s)
{
    const int L = s->L;
    /* near field: |b0(j) - b0(i)| <= 1 */
    for (int64_t j = 0; j < n; ++j)
        s->label[j] = (iabs64(j / r - i / r) <= 1) ? 0 : -1;
    /* far field, level by level: |b_l(j) - b_l(i)| <= 1 and not yet assigned */
    for (int l = 1; l < L; ++l) {
        int64_t blk = r << l; /* r * 2^l */
        for (int64_t j = 0; j < n; ++j)
            if (s->label[j] < 0 && iabs64(j / blk - i / blk) <= 1) s->label[j] = (int8_t)l;
    }
    /* the sets must cover [n] */
    for (int64_t j = 0; j < n; ++j)
        if (s->label[j] < 0) return FMAO_ERR_COVER;
    /* G_l(i): level-l groups that lie entirely inside F_l(i) */
    for (int l = 1; l < L; ++l) {
        int64_t len = group_len(r, l);
        int64_t M = ceil_div(n, len);
        int64_t cnt = 0, covered = 0, inF = 0;
        for (int64_t m = 0; m < M; ++m) {
            int64_t a = m * len, e = a + len < n ? a + len : n;
            int inside = 1;
            for (int64_t j = a; j < e; ++j)
                if (s->label[j] != l) { inside = 0; break; }
            if (inside) {
                s->grp[(int64_t)l * s->gcap + cnt++] = m;
                covered += e - a;
            }
        }
        for (int64_t j = 0; j < n; ++j) inF += (s->label[j] == l);
        /* F_l(i) must be exactly the union of the listed groups */
        if (covered != inF) return FMAO_ERR_COVER;
        s->ngrp[l] = cnt;
    }
    return FMAO_OK;
}

/* Export of the per-base-block lists for tests: out[b][l-1][k], k < kcap,
 * ascending group index, padded with -1.  near_lo/near_hi receive the first
 * and one-past-last token of N(i).  Returns FMAO_ERR_ARG when a list is
 * longer than kcap. */
int fmao_lists_1d(int64_t n, int64_t r, int32_t kcap, int32_t *out,
                  int64_t *near_lo, int64_t *near_hi)
{
    if (r <= 0 || n <= 0 || n % r || kcap <= 0) return FMAO_ERR_ARG;
    const int64_t nb = n / r;
    const int L = fmao_num_levels(nb);
    int rc = FMAO_OK;
    sets_t s;
    if (sets_alloc(&s, n, L)) { sets_free(&s); return FMAO_ERR_ALLOC; }
    for (int64_t b = 0; b < nb && rc == FMAO_OK; ++b) {
        rc = build_sets_1d(n, r, b * r, &s);
        if (rc) break;
        int64_t lo = -1, hi = -1;
        for (int64_t j = 0; j < n; ++j)
            if (s.label[j] == 0) { if (lo < 0) lo = j; hi = j + 1; }
        if (near_lo) near_lo[b] = lo;
        if (near_hi) near_hi[b] = hi;
        for (int l = 1; l < L; ++l) {
            int32_t *o = out + (b * (L - 1) + (l - 1)) * kcap;
            if (s.ngrp[l] > kcap) { rc = FMAO_ERR_ARG; break; }
            for (int32_t k = 0; k < kcap; ++k)
                o[k] = k < s.ngrp[l] ? (int32_t)s.grp[(int64_t)l * s.gcap + k] : -1;
        }
    }
    sets_free(&s);
    return rc;
}

/* ------------------------------------------------------------------ */
/* 1D coarsening (Eq. agg1d), every level directly from the fine tokens */
/* pi: level l, basis s at offset p*r*(2^(l-1)-1) + s*len, len =        */
/* r*2^(l-1).  out: [p*R][d], level l at row offset p*sum_{l'<l} M_l',  */
/* basis s, group m at row s*M_l + m within the level.                  */
/* ------------------------------------------------------------------ */
static void coarsen_1d(const double *x, int64_t n, int64_t d, int64_t r, int L,
                       const double *pi, int64_t p, double *out)
{
    int64_t row = 0;
    for (int l = 1; l < L; ++l) {
        int64_t len = group_len(r, l);
        int64_t M = ceil_div(n, len);
        for (int64_t b = 0; b < p; ++b)
            for (int64_t m = 0; m < M; ++m, ++row) {
                const double *w = pi + p * r * ((1LL << (l - 1)) - 1) + b * len;
                double *o = out + row * d;
                for (int64_t c = 0; c < d; ++c) o[c] = 0.0;
                for (int64_t j = m * len; j < (m + 1) * len && j < n; ++j)
                    for (int64_t c = 0; c < d; ++c) o[c] += w[j - m * len] * x[j * d + c];
            }
    }
}

int fmao_coarsen_1d(const double *x, int64_t n, int64_t d, int64_t r, int64_t p,
                    const double *pi, double *out)
{
    if (!x || !pi || !out || r <= 0 || n <= 0 || n % r || d <= 0 || p < 1) return FMAO_ERR_ARG;
    coarsen_1d(x, n, d, r, fmao_num_levels(n / r), pi, p, out);
    return FMAO_OK;
}

/* ------------------------------------------------------------------ */
/* Attention for one query row over an explicit source list.           */
/* Sources are either fine tokens (pointer into K/V) or coarse rows.   */
/* set_id groups sources for the per-set normalisation (0 = near,      */
/* l = level l).                                                        */
/* ------------------------------------------------------------------ */
typedef struct {
    const double *k;
    const double *v;
    int set_id;
    const double *q;   /* query that scores this source (NULL: the row's own) */
} src_t;

static void attend_row(const double *q, const src_t *src, int64_t ns, int64_t d,
                       double scale, int norm_mode, int nsets, double *score, double *out)
{
    for (int64_t c = 0; c < d; ++c) out[c] = 0.0;
    for (int64_t t = 0; t < ns; ++t) {
        double acc = 0.0;
        const double *qq = src[t].q ? src[t].q : q;
        for (int64_t c = 0; c < d; ++c) acc += qq[c] * src[t].k[c];
        score[t] = scale * acc;
    }
    if (norm_mode == 0) {
        /* one softmax over every source of the row */
        double mx = -INFINITY, z = 0.0;
        for (int64_t t = 0; t < ns; ++t) mx = score[t] > mx ? score[t] : mx;
        for (int64_t t = 0; t < ns; ++t) z += exp(score[t] - mx);
        for (int64_t t = 0; t < ns; ++t) {
            double w = exp(score[t] - mx) / z;
            for (int64_t c = 0; c < d; ++c) out[c] += w * src[t].v[c];
        }
    } else {
        /* printed form: alpha normalised over N(i), beta^l over G_l(i) */
        for (int set = 0; set < nsets; ++set) {
            double mx = -INFINITY, z = 0.0;
            int any = 0;
            for (int64_t t = 0; t < ns; ++t)
                if (src[t].set_id == set) { any = 1; mx = score[t] > mx ? score[t] : mx; }
            if (!any) continue;
            for (int64_t t = 0; t < ns; ++t)
                if (src[t].set_id == set) z += exp(score[t] - mx);
            for (int64_t t = 0; t < ns; ++t)
                if (src[t].set_id == set) {
                    double w = exp(score[t] - mx) / z;
                    for (int64_t c = 0; c < d; ++c) out[c] += w * src[t].v[c];
                }
        }
    }
}

/* ------------------------------------------------------------------ */
/* 1D forward for a batch of independent (batch, head) slices.         */
/*   q, k, v, o : [S][n][d] row-major, S = number of slices           */
/*   pik, piv   : [S or 1][wlen] (w_stride = 0 shares one set)        */
/*   counts     : optional [S][n], number of sources of every row      */
/* ------------------------------------------------------------------ */
int fmao_forward_1d(const double *q, const double *k, const double *v,
                    int64_t S, int64_t n, int64_t d, int64_t r, int causal, int64_t p,
                    const double *pik, const double *piv, const double *piq, int64_t w_stride,
                    double scale, int norm_mode, double *o, int64_t *counts)
{
    if (!q || !k || !v || !o || S < 0 || r <= 0 || n <= 0 || n % r || d <= 0 || p < 1) return FMAO_ERR_ARG;
    if (piq && (causal || p != 1)) return FMAO_ERR_ARG;   /* FMA-linear: bidirectional, rank 1 */
    const int64_t nb = n / r;
    const int L = fmao_num_levels(nb);
    if (L > 1 && (!pik || !piv)) return FMAO_ERR_ARG;
    const int64_t R = p * fmao_coarse_rows_1d(n, r);
    int err = FMAO_OK;

    /* coarse keys and values (and FMA-linear: queries) of every slice, Eq. agg1d */
    const size_t cbytes = sizeof(double) * (size_t)((S * R > 0 ? S * R : 1) * d);
    double *kbar = (double *)malloc(cbytes);
    double *vbar = (double *)malloc(cbytes);
    double *qbar = piq ? (double *)malloc(cbytes) : NULL;
    if (!kbar || !vbar || (piq && !qbar)) { free(kbar); free(vbar); free(qbar); return FMAO_ERR_ALLOC; }
    if (L > 1) {
        #pragma omp parallel for schedule(dynamic, 1)
        for (int64_t sl = 0; sl < S; ++sl) {
            coarsen_1d(k + sl * n * d, n, d, r, L, pik + sl * w_stride, p, kbar + sl * R * d);
            coarsen_1d(v + sl * n * d, n, d, r, L, piv + sl * w_stride, p, vbar + sl * R * d);
            if (piq) coarsen_1d(q + sl * n * d, n, d, r, L, piq + sl * w_stride, p, qbar + sl * R * d);
        }
    }

    #pragma omp parallel
    {
        sets_t s;
        int local_err = sets_alloc(&s, n, L);
        int64_t cap = n + R + 1;
        src_t *src = (src_t *)malloc(sizeof(src_t) * (size_t)cap);
        int64_t *near = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
        double *score = (double *)malloc(sizeof(double) * (size_t)cap);
        if (!src || !near || !score) local_err = FMAO_ERR_ALLOC;

        #pragma omp for schedule(dynamic, 1)
        for (int64_t b = 0; b < nb; ++b) {
            if (local_err) continue;
            /* the sets of every row of base block b (they depend on b only) */
            int rc = build_sets_1d(n, r, b * r, &s);
            if (rc) { local_err = rc; continue; }
            int64_t nnear = 0;
            for (int64_t j = 0; j < n; ++j)
                if (s.label[j] == 0) near[nnear++] = j;
            for (int64_t sl = 0; sl < S; ++sl) {
                const double *qs = q + sl * n * d, *ks = k + sl * n * d, *vs = v + sl * n * d;
                const double *kb = kbar + sl * R * d, *vb = vbar + sl * R * d;
                const double *qbs = qbar ? qbar + sl * R * d : NULL;
                for (int64_t i = b * r; i < (b + 1) * r; ++i) {
                    int64_t ns = 0;
                    for (int64_t t = 0; t < nnear; ++t) {
                        int64_t j = near[t];
                        if (!causal || j <= i) src[ns++] = (src_t){ks + j * d, vs + j * d, 0, NULL};
                    }
                    int64_t off = 0;
                    for (int l = 1; l < L; ++l) {
                        int64_t len = group_len(r, l);
                        for (int64_t t = 0; t < s.ngrp[l]; ++t) {
                            int64_t m = s.grp[(int64_t)l * s.gcap + t];
                            int64_t last = (m + 1) * len < n ? (m + 1) * len - 1 : n - 1;
                            /* FMA-linear: the coarse query of the row's own level-l group */
                            const double *cq = qbs ? qbs + (off + i / len) * d : NULL;
                            if (!causal || last <= i)
                                for (int64_t b = 0; b < p; ++b) {
                                    const int64_t row = off + b * ceil_div(n, len) + m;
                                    src[ns++] = (src_t){kb + row * d, vb + row * d, l, cq};
                                }
                        }
                        off += p * ceil_div(n, len);
                    }
                    attend_row(qs + i * d, src, ns, d, scale, norm_mode, L > 0 ? L : 1, score,
                               o + (sl * n + i) * d);
                    if (counts) counts[sl * n + i] = ns;
                }
            }
        }
        if (local_err) {
            #pragma omp critical
            err = local_err;
        }
        sets_free(&s);
        free(src);
        free(near);
        free(score);
    }
    free(kbar);
    free(vbar);
    free(qbar);
    return err;
}

/* ------------------------------------------------------------------ */
/* 2D (Sec. 3, "FMA in 2D").  Token t = x*W + y, x = row.              */
/* ------------------------------------------------------------------ */
static int build_sets_2d(int64_t H, int64_t W, int64_t r, int64_t xi, int64_t yi, sets_t *s)
{
    const int L = s->L;
    const int64_t n = H * W;
    for (int64_t t = 0; t < n; ++t) {
        int64_t x = t / W, y = t % W;
        s->label[t] = (iabs64(x / r - xi / r) <= 1 && iabs64(y / r - yi / r) <= 1) ? 0 : -1;
    }
    for (int l = 1; l < L; ++l) {
        int64_t blk = r << l;
        for (int64_t t = 0; t < n; ++t) {
            int64_t x = t / W, y = t % W;
            if (s->label[t] < 0 && iabs64(x / blk - xi / blk) <= 1 && iabs64(y / blk - yi / blk) <= 1)
                s->label[t] = (int8_t)l;
        }
    }
    for (int64_t t = 0; t < n; ++t)
        if (s->label[t] < 0) return FMAO_ERR_COVER;
    for (int l = 1; l < L; ++l) {
        int64_t len = group_len(r, l);
        int64_t Mx = ceil_div(H, len), My = ceil_div(W, len);
        int64_t cnt = 0, covered = 0, inF = 0;
        for (int64_t u = 0; u < Mx; ++u)
            for (int64_t vv = 0; vv < My; ++vv) {
                int inside = 1;
                int64_t area = 0;
                for (int64_t x = u * len; x < (u + 1) * len && x < H && inside; ++x)
                    for (int64_t y = vv * len; y < (vv + 1) * len && y < W; ++y) {
                        if (s->label[x * W + y] != l) { inside = 0; break; }
                        ++area;
                    }
                if (inside) {
                    s->grp[(int64_t)l * s->gcap + cnt++] = u * My + vv;
                    covered += area;
                }
            }
        for (int64_t t = 0; t < n; ++t) inF += (s->label[t] == l);
        if (covered != inF) return FMAO_ERR_COVER;
        s->ngrp[l] = cnt;
    }
    return FMAO_OK;
}

int fmao_lists_2d_hw(int64_t H, int64_t W, int64_t r, int32_t kcap, int32_t *out)
{
    if (r <= 0 || W <= 0 || H <= 0 || W % r || H % r || kcap <= 0) return FMAO_ERR_ARG;
    const int64_t nbx = H / r, nby = W / r;
    const int L = levels_2d(H, W, r);
    int rc = FMAO_OK;
    sets_t s;
    if (sets_alloc(&s, H * W, L)) { sets_free(&s); return FMAO_ERR_ALLOC; }
    for (int64_t cx = 0; cx < nbx && rc == FMAO_OK; ++cx)
        for (int64_t cy = 0; cy < nby && rc == FMAO_OK; ++cy) {
            rc = build_sets_2d(H, W, r, cx * r, cy * r, &s);
            if (rc) break;
            int64_t cell = cx * nby + cy;
            for (int l = 1; l < L; ++l) {
                int32_t *o = out + (cell * (L - 1) + (l - 1)) * kcap;
                if (s.ngrp[l] > kcap) { rc = FMAO_ERR_ARG; break; }
                for (int32_t t = 0; t < kcap; ++t)
                    o[t] = t < s.ngrp[l] ? (int32_t)s.grp[(int64_t)l * s.gcap + t] : -1;
            }
        }
    sets_free(&s);
    return rc;
}

int fmao_lists_2d(int64_t W, int64_t r, int32_t kcap, int32_t *out) { return fmao_lists_2d_hw(W, W, r, kcap, out); }

/* 2D coarsening (Eq. agg2d): full double sum with Pi[a][b] = pi_x[a]*pi_y[b].
 * pi: level l, basis s at offset p*2r*(2^(l-1)-1) + s*2*len:
 * [pi_x (len) | pi_y (len)].  out rows: level offset + s*M_l^2 + u*M_l + v. */
static void coarsen_2d(const double *x, int64_t H, int64_t W, int64_t d, int64_t r, int L,
                       const double *pi, int64_t p, double *out)
{
    int64_t row = 0;
    for (int l = 1; l < L; ++l) {
        int64_t len = group_len(r, l);
        int64_t Mx = ceil_div(H, len), My = ceil_div(W, len);
        for (int64_t b = 0; b < p; ++b)
            for (int64_t u = 0; u < Mx; ++u)
                for (int64_t vv = 0; vv < My; ++vv, ++row) {
                    const double *px = pi + p * 2 * r * ((1LL << (l - 1)) - 1) + b * 2 * len;
                    const double *py = px + len;
                    double *o = out + row * d;
                    for (int64_t c = 0; c < d; ++c) o[c] = 0.0;
                    for (int64_t a = 0; a < len && u * len + a < H; ++a)
                        for (int64_t bb = 0; bb < len && vv * len + bb < W; ++bb) {
                            double w = px[a] * py[bb];
                            const double *src = x + ((u * len + a) * W + (vv * len + bb)) * d;
                            for (int64_t c = 0; c < d; ++c) o[c] += w * src[c];
                        }
                }
    }
}

int fmao_coarsen_2d_hw(const double *x, int64_t H, int64_t W, int64_t d, int64_t r, int64_t p,
                       const double *pi, double *out)
{
    if (!x || !pi || !out || r <= 0 || W <= 0 || H <= 0 || W % r || H % r || d <= 0 || p < 1) return FMAO_ERR_ARG;
    coarsen_2d(x, H, W, d, r, levels_2d(H, W, r), pi, p, out);
    return FMAO_OK;
}

int fmao_coarsen_2d(const double *x, int64_t W, int64_t d, int64_t r, int64_t p, const double *pi, double *out)
{
    return fmao_coarsen_2d_hw(x, W, W, d, r, p, pi, out);
}

int fmao_forward_2d_hw(const double *q, const double *k, const double *v,
                       int64_t S, int64_t H, int64_t W, int64_t d, int64_t r, int64_t p,
                       const double *pik, const double *piv, const double *piq, int64_t w_stride,
                       double scale, int norm_mode, double *o, int64_t *counts)
{
    if (!q || !k || !v || !o || S < 0 || r <= 0 || W <= 0 || H <= 0 || W % r || H % r || d <= 0 || p < 1)
        return FMAO_ERR_ARG;
    if (piq && p != 1) return FMAO_ERR_ARG;   /* FMA-linear: rank 1 */
    const int64_t n = H * W;
    const int64_t nbx = H / r, nby = W / r;
    const int L = levels_2d(H, W, r);
    if (L > 1 && (!pik || !piv)) return FMAO_ERR_ARG;
    const int64_t R = p * fmao_coarse_rows_2d_hw(H, W, r);
    const int64_t ncell = nbx * nby;
    int err = FMAO_OK;

    /* coarse keys and values (and FMA-linear: queries) of every slice, Eq. agg2d */
    const size_t cbytes = sizeof(double) * (size_t)((S * R > 0 ? S * R : 1) * d);
    double *kbar = (double *)malloc(cbytes);
    double *vbar = (double *)malloc(cbytes);
    double *qbar = piq ? (double *)malloc(cbytes) : NULL;
    if (!kbar || !vbar || (piq && !qbar)) { free(kbar); free(vbar); free(qbar); return FMAO_ERR_ALLOC; }
    if (L > 1) {
        #pragma omp parallel for schedule(dynamic, 1)
        for (int64_t sl = 0; sl < S; ++sl) {
            coarsen_2d(k + sl * n * d, H, W, d, r, L, pik + sl * w_stride, p, kbar + sl * R * d);
            coarsen_2d(v + sl * n * d, H, W, d, r, L, piv + sl * w_stride, p, vbar + sl * R * d);
            if (piq) coarsen_2d(q + sl * n * d, H, W, d, r, L, piq + sl * w_stride, p, qbar + sl * R * d);
        }
    }

    #pragma omp parallel
    {
        sets_t s;
        int local_err = sets_alloc(&s, n, L);
        int64_t cap = n + R + 1;
        src_t *src = (src_t *)malloc(sizeof(src_t) * (size_t)cap);
        double *score = (double *)malloc(sizeof(double) * (size_t)cap);
        if (!src || !score) local_err = FMAO_ERR_ALLOC;

        #pragma omp for schedule(dynamic, 1)
        for (int64_t cell = 0; cell < ncell; ++cell) {
            if (local_err) continue;
            int64_t cx = cell / nby, cy = cell % nby;
            int rc = build_sets_2d(H, W, r, cx * r, cy * r, &s);
            if (rc) { local_err = rc; continue; }
            for (int64_t sl = 0; sl < S; ++sl) {
                const double *qs = q + sl * n * d, *ks = k + sl * n * d, *vs = v + sl * n * d;
                const double *kb = kbar + sl * R * d, *vb = vbar + sl * R * d;
                const double *qbs = qbar ? qbar + sl * R * d : NULL;
                int64_t ns = 0;
                for (int64_t t = 0; t < n; ++t)
                    if (s.label[t] == 0) src[ns++] = (src_t){ks + t * d, vs + t * d, 0, NULL};
                int64_t off = 0;
                for (int l = 1; l < L; ++l) {
                    const int64_t len = group_len(r, l);
                    const int64_t Mx = ceil_div(H, len), My = ceil_div(W, len);
                    /* FMA-linear: the coarse query of the cell's own level-l square */
                    const double *cq = qbs ? qbs + (off + (cx * r / len) * My + (cy * r / len)) * d : NULL;
                    for (int64_t t = 0; t < s.ngrp[l]; ++t) {
                        int64_t g = s.grp[(int64_t)l * s.gcap + t];
                        for (int64_t b = 0; b < p; ++b) {
                            const int64_t row = off + b * Mx * My + g;
                            src[ns++] = (src_t){kb + row * d, vb + row * d, l, cq};
                        }
                    }
                    off += p * Mx * My;
                }
                for (int64_t x = cx * r; x < (cx + 1) * r; ++x)
                    for (int64_t y = cy * r; y < (cy + 1) * r; ++y) {
                        int64_t i = x * W + y;
                        attend_row(qs + i * d, src, ns, d, scale, norm_mode, L > 0 ? L : 1, score,
                                   o + (sl * n + i) * d);
                        if (counts) counts[sl * n + i] = ns;
                    }
            }
        }
        if (local_err) {
            #pragma omp critical
            err = local_err;
        }
        sets_free(&s);
        free(src);
        free(score);
    }
    free(kbar);
    free(vbar);
    free(qbar);
    return err;
}

int fmao_forward_2d(const double *q, const double *k, const double *v, int64_t S, int64_t W, int64_t d, int64_t r,
                    int64_t p, const double *pik, const double *piv, const double *piq, int64_t w_stride,
                    double scale, int norm_mode, double *o, int64_t *counts)
{
    return fmao_forward_2d_hw(q, k, v, S, W, W, d, r, p, pik, piv, piq, w_stride, scale, norm_mode, o, counts);
}

/* Label export for tests: label[j] (0 = near, l = level-l far) for query row i. */
int fmao_labels_1d(int64_t n, int64_t r, int64_t i, int8_t *label)
{
    if (!label || r <= 0 || n <= 0 || n % r || i < 0 || i >= n) return FMAO_ERR_ARG;
    sets_t s;
    int rc = sets_alloc(&s, n, fmao_num_levels(n / r));
    if (!rc) rc = build_sets_1d(n, r, i, &s);
    if (!rc) memcpy(label, s.label, (size_t)n);
    sets_free(&s);
    return rc;
}

int fmao_labels_2d_hw(int64_t H, int64_t W, int64_t r, int64_t i, int8_t *label)
{
    if (!label || r <= 0 || W <= 0 || H <= 0 || W % r || H % r || i < 0 || i >= H * W) return FMAO_ERR_ARG;
    sets_t s;
    int rc = sets_alloc(&s, H * W, levels_2d(H, W, r));
    if (!rc) rc = build_sets_2d(H, W, r, i / W, i % W, &s);
    if (!rc) memcpy(label, s.label, (size_t)(H * W));
    sets_free(&s);
    return rc;
}

int fmao_labels_2d(int64_t W, int64_t r, int64_t i, int8_t *label) { return fmao_labels_2d_hw(W, W, r, i, label); }


/* ================================================================== */
/* Backward pass.                                                      */
/* ================================================================== */

/* one source of a row for the backward pass: a fine token (coarse = 0) or
 * a coarse row, index into the slice's rows, set id as in attend_row; qidx:
 * FMA-linear, the coarse query (row of the slice's coarse queries) that
 * scores this source, -1 for the row's own query */
typedef struct {
    int64_t idx;
    int coarse;
    int set_id;
    int64_t qidx;
} bsrc_t;

/* Gradients of one row: forward probabilities, dS, and the accumulation into
 * dq (this row), dk/dv (fine rows) and dkb/dvb (coarse rows). */
static void backward_row(const double *qi, const double *doi, const bsrc_t *src, int64_t ns, int64_t d,
                         const double *ks, const double *vs, const double *kb, const double *vb,
                         const double *qb, double scale, int norm_mode, int nsets, double *score, double *prob,
                         double *dpv, double *dqi, double *dks, double *dvs, double *dkb, double *dvb,
                         double *dqb)
{
    for (int64_t t = 0; t < ns; ++t) {
        const double *kt = src[t].coarse ? kb + src[t].idx * d : ks + src[t].idx * d;
        const double *vt = src[t].coarse ? vb + src[t].idx * d : vs + src[t].idx * d;
        const double *qq = src[t].qidx >= 0 ? qb + src[t].qidx * d : qi;
        double acc = 0.0, dp = 0.0;
        for (int64_t c = 0; c < d; ++c) {
            acc += qq[c] * kt[c];
            dp += doi[c] * vt[c];
        }
        score[t] = scale * acc;
        dpv[t] = dp;   /* dP_t = dO . v_t */
    }
    /* probabilities, then D per normalisation set */
    const int nset_eff = norm_mode == 0 ? 1 : nsets;
    for (int set = 0; set < nset_eff; ++set) {
        double mx = -INFINITY, z = 0.0, dsum = 0.0;
        int any = 0;
        for (int64_t t = 0; t < ns; ++t)
            if (norm_mode == 0 || src[t].set_id == set) { any = 1; mx = score[t] > mx ? score[t] : mx; }
        if (!any) continue;
        for (int64_t t = 0; t < ns; ++t)
            if (norm_mode == 0 || src[t].set_id == set) z += exp(score[t] - mx);
        for (int64_t t = 0; t < ns; ++t)
            if (norm_mode == 0 || src[t].set_id == set) {
                prob[t] = exp(score[t] - mx) / z;
                dsum += prob[t] * dpv[t];
            }
        for (int64_t t = 0; t < ns; ++t)
            if (norm_mode == 0 || src[t].set_id == set) dpv[t] = prob[t] * (dpv[t] - dsum);   /* now dS_t */
    }
    for (int64_t t = 0; t < ns; ++t) {
        const double *kt = src[t].coarse ? kb + src[t].idx * d : ks + src[t].idx * d;
        double *dkt = src[t].coarse ? dkb + src[t].idx * d : dks + src[t].idx * d;
        double *dvt = src[t].coarse ? dvb + src[t].idx * d : dvs + src[t].idx * d;
        /* the query that scored the source receives its gradient */
        const double *qq = src[t].qidx >= 0 ? qb + src[t].qidx * d : qi;
        double *dqq = src[t].qidx >= 0 ? dqb + src[t].qidx * d : dqi;
        for (int64_t c = 0; c < d; ++c) {
            dqq[c] += scale * dpv[t] * kt[c];
            dkt[c] += scale * dpv[t] * qq[c];
            dvt[c] += prob[t] * doi[c];
        }
    }
}

/* Coarsening backward, 1D: x and its gradient dx, pi and its gradient dpi
 * (same layouts as coarsen_1d), dbar = gradient of the coarse rows. */
static void coarsen_1d_backward(const double *x, int64_t n, int64_t d, int64_t r, int L, const double *pi,
                                int64_t p, const double *dbar, double *dx, double *dpi)
{
    int64_t row = 0;
    for (int l = 1; l < L; ++l) {
        int64_t len = group_len(r, l);
        int64_t M = ceil_div(n, len);
        for (int64_t b = 0; b < p; ++b)
            for (int64_t m = 0; m < M; ++m, ++row) {
                const int64_t woff = p * r * ((1LL << (l - 1)) - 1) + b * len;
                const double *g = dbar + row * d;
                for (int64_t j = m * len; j < (m + 1) * len && j < n; ++j) {
                    double dot = 0.0;
                    for (int64_t c = 0; c < d; ++c) {
                        dx[j * d + c] += pi[woff + j - m * len] * g[c];
                        dot += x[j * d + c] * g[c];
                    }
                    dpi[woff + j - m * len] += dot;
                }
            }
    }
}

/* Coarsening backward, 2D: Pi[a][b] = pi_x[a] * pi_y[b]. */
static void coarsen_2d_backward(const double *x, int64_t H, int64_t W, int64_t d, int64_t r, int L,
                                const double *pi, int64_t p, const double *dbar, double *dx, double *dpi)
{
    int64_t row = 0;
    for (int l = 1; l < L; ++l) {
        int64_t len = group_len(r, l);
        int64_t Mx = ceil_div(H, len), My = ceil_div(W, len);
        for (int64_t b = 0; b < p; ++b)
            for (int64_t u = 0; u < Mx; ++u)
                for (int64_t vv = 0; vv < My; ++vv, ++row) {
                    const int64_t woff = p * 2 * r * ((1LL << (l - 1)) - 1) + b * 2 * len;
                    const double *px = pi + woff, *py = px + len;
                    double *dpx = dpi + woff, *dpy = dpx + len;
                    const double *g = dbar + row * d;
                    for (int64_t a = 0; a < len && u * len + a < H; ++a)
                        for (int64_t bb = 0; bb < len && vv * len + bb < W; ++bb) {
                            const int64_t t = (u * len + a) * W + (vv * len + bb);
                            double dot = 0.0;
                            for (int64_t c = 0; c < d; ++c) {
                                dx[t * d + c] += px[a] * py[bb] * g[c];
                                dot += x[t * d + c] * g[c];
                            }
                            dpx[a] += py[bb] * dot;
                            dpy[bb] += px[a] * dot;
                        }
                }
    }
}

/* ------------------------------------------------------------------ */
/* 1D / 2D backward for a batch of slices.                             */
/*   dout        : [S][n][d] upstream gradient of the output           */
/*   dq, dk, dv  : [S][n][d] (overwritten)                             */
/*   dpik, dpiv  : [S][wlen] per-slice weight gradients (overwritten);  */
/*                 slices that share a weight set add theirs up        */
/* Slices run in parallel; inside a slice everything is sequential.    */
/* ------------------------------------------------------------------ */
static int backward_common(int two_d, const double *q, const double *k, const double *v, int64_t S, int64_t n,
                           int64_t W, int64_t d, int64_t r, int causal, int64_t p, const double *pik,
                           const double *piv, const double *piq, int64_t w_stride, double scale, int norm_mode,
                           const double *dout, double *dq, double *dk, double *dv, double *dpik, double *dpiv,
                           double *dpiq)
{
    const int64_t H = two_d ? n / W : 0;
    const int64_t ratio = two_d ? (H > W ? H : W) / r : n / r;
    const int L = fmao_num_levels(ratio);
    if (L > 1 && (!pik || !piv || !dpik || !dpiv)) return FMAO_ERR_ARG;
    /* FMA-linear: bidirectional, rank 1, joint normalisation */
    if (piq && (causal || p != 1 || norm_mode != 0 || (L > 1 && !dpiq))) return FMAO_ERR_ARG;
    const int lin = piq != NULL && L > 1;
    const int64_t R1 = two_d ? fmao_coarse_rows_2d_hw(H, W, r) : fmao_coarse_rows_1d(n, r);
    const int64_t R = p * R1;
    const int64_t wlen = L > 1 ? p * (two_d ? 2 : 1) * r * ((1LL << (L - 1)) - 1) : 0;
    const int64_t nby = two_d ? W / r : 0;
    const int64_t nblk = two_d ? (H / r) * nby : ratio;
    int err = FMAO_OK;
    memset(dq, 0, sizeof(double) * (size_t)(S * n * d));
    memset(dk, 0, sizeof(double) * (size_t)(S * n * d));
    memset(dv, 0, sizeof(double) * (size_t)(S * n * d));
    if (wlen) {
        memset(dpik, 0, sizeof(double) * (size_t)(S * wlen));
        memset(dpiv, 0, sizeof(double) * (size_t)(S * wlen));
        if (lin) memset(dpiq, 0, sizeof(double) * (size_t)(S * wlen));
    }

    #pragma omp parallel
    {
        sets_t s;
        int local_err = sets_alloc(&s, n, L);
        const int64_t cap = n + R + 1;
        bsrc_t *src = (bsrc_t *)malloc(sizeof(bsrc_t) * (size_t)cap);
        double *score = (double *)malloc(sizeof(double) * (size_t)cap);
        double *prob = (double *)malloc(sizeof(double) * (size_t)cap);
        double *dpv = (double *)malloc(sizeof(double) * (size_t)cap);
        const size_t cb = sizeof(double) * (size_t)((R > 0 ? R : 1) * d);
        double *kbar = (double *)malloc(cb), *vbar = (double *)malloc(cb);
        double *dkbar = (double *)malloc(cb), *dvbar = (double *)malloc(cb);
        double *qbar = (double *)malloc(cb), *dqbar = (double *)malloc(cb);
        if (!src || !score || !prob || !dpv || !kbar || !vbar || !dkbar || !dvbar || !qbar || !dqbar)
            local_err = FMAO_ERR_ALLOC;

        #pragma omp for schedule(dynamic, 1)
        for (int64_t sl = 0; sl < S; ++sl) {
            if (local_err) continue;
            const double *qs = q + sl * n * d, *ks = k + sl * n * d, *vs = v + sl * n * d;
            const double *dos = dout + sl * n * d;
            double *dqs = dq + sl * n * d, *dks = dk + sl * n * d, *dvs = dv + sl * n * d;
            memset(dkbar, 0, cb);
            memset(dvbar, 0, cb);
            memset(dqbar, 0, cb);
            if (L > 1) {
                if (two_d) {
                    coarsen_2d(ks, H, W, d, r, L, pik + sl * w_stride, p, kbar);
                    coarsen_2d(vs, H, W, d, r, L, piv + sl * w_stride, p, vbar);
                    if (lin) coarsen_2d(qs, H, W, d, r, L, piq + sl * w_stride, p, qbar);
                } else {
                    coarsen_1d(ks, n, d, r, L, pik + sl * w_stride, p, kbar);
                    coarsen_1d(vs, n, d, r, L, piv + sl * w_stride, p, vbar);
                    if (lin) coarsen_1d(qs, n, d, r, L, piq + sl * w_stride, p, qbar);
                }
            }
            for (int64_t b = 0; b < nblk && !local_err; ++b) {
                int rc;
                if (two_d)
                    rc = build_sets_2d(H, W, r, (b / nby) * r, (b % nby) * r, &s);
                else
                    rc = build_sets_1d(n, r, b * r, &s);
                if (rc) { local_err = rc; break; }
                for (int64_t e = 0; e < r * (two_d ? r : 1); ++e) {
                    const int64_t i = two_d ? ((b / nby) * r + e / r) * W + (b % nby) * r + e % r : b * r + e;
                    int64_t ns = 0;
                    for (int64_t j = 0; j < n; ++j)
                        if (s.label[j] == 0 && (!causal || j <= i)) src[ns++] = (bsrc_t){j, 0, 0, -1};
                    int64_t off = 0;
                    for (int l = 1; l < L; ++l) {
                        const int64_t len = group_len(r, l);
                        const int64_t My = two_d ? ceil_div(W, len) : ceil_div(n, len);
                        const int64_t M = two_d ? ceil_div(H, len) * My : My;
                        /* FMA-linear: the coarse query of the row's own level-l group */
                        const int64_t qg = !lin ? -1 : two_d ? off + ((i / W) / len) * My + (i % W) / len
                                                             : off + i / len;
                        for (int64_t t = 0; t < s.ngrp[l]; ++t) {
                            const int64_t m = s.grp[(int64_t)l * s.gcap + t];
                            const int64_t last = (m + 1) * len < n ? (m + 1) * len - 1 : n - 1;
                            if (two_d || !causal || last <= i)
                                for (int64_t bb = 0; bb < p; ++bb)
                                    src[ns++] = (bsrc_t){off + bb * M + m, 1, l, qg};
                        }
                        off += p * M;
                    }
                    backward_row(qs + i * d, dos + i * d, src, ns, d, ks, vs, kbar, vbar, qbar, scale, norm_mode,
                                 L > 0 ? L : 1, score, prob, dpv, dqs + i * d, dks, dvs, dkbar, dvbar, dqbar);
                }
            }
            if (L > 1 && !local_err) {
                if (two_d) {
                    coarsen_2d_backward(ks, H, W, d, r, L, pik + sl * w_stride, p, dkbar, dks, dpik + sl * wlen);
                    coarsen_2d_backward(vs, H, W, d, r, L, piv + sl * w_stride, p, dvbar, dvs, dpiv + sl * wlen);
                    if (lin)
                        coarsen_2d_backward(qs, H, W, d, r, L, piq + sl * w_stride, p, dqbar, dqs, dpiq + sl * wlen);
                } else {
                    coarsen_1d_backward(ks, n, d, r, L, pik + sl * w_stride, p, dkbar, dks, dpik + sl * wlen);
                    coarsen_1d_backward(vs, n, d, r, L, piv + sl * w_stride, p, dvbar, dvs, dpiv + sl * wlen);
                    if (lin) coarsen_1d_backward(qs, n, d, r, L, piq + sl * w_stride, p, dqbar, dqs, dpiq + sl * wlen);
                }
            }
        }
        if (local_err) {
            #pragma omp critical
            err = local_err;
        }
        sets_free(&s);
        free(src);
        free(score);
        free(prob);
        free(dpv);
        free(kbar);
        free(vbar);
        free(dkbar);
        free(dvbar);
        free(qbar);
        free(dqbar);
    }
    return err;
}

int fmao_backward_1d(const double *q, const double *k, const double *v, int64_t S, int64_t n, int64_t d,
                     int64_t r, int causal, int64_t p, const double *pik, const double *piv, int64_t w_stride,
                     double scale, int norm_mode, const double *dout, double *dq, double *dk, double *dv,
                     double *dpik, double *dpiv)
{
    if (!q || !k || !v || !dout || !dq || !dk || !dv || S < 0 || r <= 0 || n <= 0 || n % r || d <= 0 || p < 1)
        return FMAO_ERR_ARG;
    return backward_common(0, q, k, v, S, n, 0, d, r, causal, p, pik, piv, NULL, w_stride, scale, norm_mode, dout,
                           dq, dk, dv, dpik, dpiv, NULL);
}

int fmao_backward_2d_hw(const double *q, const double *k, const double *v, int64_t S, int64_t H, int64_t W,
                        int64_t d, int64_t r, int64_t p, const double *pik, const double *piv, int64_t w_stride,
                        double scale, int norm_mode, const double *dout, double *dq, double *dk, double *dv,
                        double *dpik, double *dpiv)
{
    if (!q || !k || !v || !dout || !dq || !dk || !dv || S < 0 || r <= 0 || W <= 0 || H <= 0 || W % r || H % r ||
        d <= 0 || p < 1)
        return FMAO_ERR_ARG;
    return backward_common(1, q, k, v, S, H * W, W, d, r, 0, p, pik, piv, NULL, w_stride, scale, norm_mode, dout,
                           dq, dk, dv, dpik, dpiv, NULL);
}

int fmao_backward_2d(const double *q, const double *k, const double *v, int64_t S, int64_t W, int64_t d,
                     int64_t r, int64_t p, const double *pik, const double *piv, int64_t w_stride, double scale,
                     int norm_mode, const double *dout, double *dq, double *dk, double *dv, double *dpik,
                     double *dpiv)
{
    return fmao_backward_2d_hw(q, k, v, S, W, W, d, r, p, pik, piv, w_stride, scale, norm_mode, dout, dq, dk, dv,
                               dpik, dpiv);
}

/* FMA-linear backward (reading R18 of the forward): the coarse sources of a
 * row are scored with the coarse query of the row's own group at their
 * level, so their score gradients flow to the coarse queries, and from there
 * through the query coarsening to q and pi^q (dpiq, [S][wlen], overwritten).
 * Bidirectional, rank 1, joint normalisation. */
int fmao_backward_linear_1d(const double *q, const double *k, const double *v, int64_t S, int64_t n, int64_t d,
                            int64_t r, const double *pik, const double *piv, const double *piq, int64_t w_stride,
                            double scale, const double *dout, double *dq, double *dk, double *dv, double *dpik,
                            double *dpiv, double *dpiq)
{
    if (!q || !k || !v || !dout || !dq || !dk || !dv || !piq || S < 0 || r <= 0 || n <= 0 || n % r || d <= 0)
        return FMAO_ERR_ARG;
    return backward_common(0, q, k, v, S, n, 0, d, r, 0, 1, pik, piv, piq, w_stride, scale, 0, dout, dq, dk, dv,
                           dpik, dpiv, dpiq);
}

int fmao_backward_linear_2d_hw(const double *q, const double *k, const double *v, int64_t S, int64_t H, int64_t W,
                               int64_t d, int64_t r, const double *pik, const double *piv, const double *piq,
                               int64_t w_stride, double scale, const double *dout, double *dq, double *dk,
                               double *dv, double *dpik, double *dpiv, double *dpiq)
{
    if (!q || !k || !v || !dout || !dq || !dk || !dv || !piq || S < 0 || r <= 0 || W <= 0 || H <= 0 || W % r ||
        H % r || d <= 0)
        return FMAO_ERR_ARG;
    return backward_common(1, q, k, v, S, H * W, W, d, r, 0, 1, pik, piv, piq, w_stride, scale, 0, dout, dq, dk,
                           dv, dpik, dpiv, dpiq);
}

int fmao_backward_linear_2d(const double *q, const double *k, const double *v, int64_t S, int64_t W, int64_t d,
                            int64_t r, const double *pik, const double *piv, const double *piq, int64_t w_stride,
                            double scale, const double *dout, double *dq, double *dk, double *dv, double *dpik,
                            double *dpiv, double *dpiq)
{
    return fmao_backward_linear_2d_hw(q, k, v, S, W, W, d, r, pik, piv, piq, w_stride, scale, dout, dq, dk, dv,
                                      dpik, dpiv, dpiq);
}
