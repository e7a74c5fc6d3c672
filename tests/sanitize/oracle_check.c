/* The C oracle under AddressSanitizer / UBSan (test infrastructure): every
 * entry point on small 1D and 2D problems, every buffer sized exactly, with
 * invariants the paper fixes checked on the results: row weights sum to 1
 * (V = 1 and value weights 1/s on every level give O = 1, Sec. 3), causal
 * outputs ignore later tokens, and the list export matches the near/far
 * cover.  Built serially (no OpenMP) so that the sanitizers see every access. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int fmao_num_levels(int64_t ratio);
int64_t fmao_coarse_rows_1d(int64_t n, int64_t r);
int64_t fmao_coarse_rows_2d(int64_t W, int64_t r);
int fmao_lists_1d(int64_t n, int64_t r, int32_t kcap, int32_t *out, int64_t *near_lo, int64_t *near_hi);
int fmao_lists_2d(int64_t W, int64_t r, int32_t kcap, int32_t *out);
int fmao_coarsen_1d(const double *x, int64_t n, int64_t d, int64_t r, int64_t p, const double *pi, double *out);
int fmao_coarsen_2d(const double *x, int64_t W, int64_t d, int64_t r, int64_t p, const double *pi, double *out);
int fmao_forward_1d(const double *q, const double *k, const double *v, int64_t S, int64_t n, int64_t d, int64_t r,
                    int causal, int64_t p, const double *pik, const double *piv, const double *piq, int64_t w_stride,
                    double scale, int norm_mode, double *o, int64_t *counts);
int fmao_forward_2d(const double *q, const double *k, const double *v, int64_t S, int64_t W, int64_t d, int64_t r,
                    int64_t p, const double *pik, const double *piv, const double *piq, int64_t w_stride,
                    double scale, int norm_mode, double *o, int64_t *counts);
int fmao_backward_1d(const double *q, const double *k, const double *v, int64_t S, int64_t n, int64_t d, int64_t r,
                     int causal, int64_t p, const double *pik, const double *piv, int64_t w_stride, double scale,
                     int norm_mode, const double *dout, double *dq, double *dk, double *dv, double *dpik,
                     double *dpiv);
int fmao_backward_2d(const double *q, const double *k, const double *v, int64_t S, int64_t W, int64_t d, int64_t r,
                     int64_t p, const double *pik, const double *piv, int64_t w_stride, double scale, int norm_mode,
                     const double *dout, double *dq, double *dk, double *dv, double *dpik, double *dpiv);

static int failures = 0;
#define CHECK(c)                                                        \
    do {                                                                \
        if (!(c)) {                                                     \
            fprintf(stderr, "FAIL line %d: %s\n", __LINE__, #c);        \
            ++failures;                                                 \
        }                                                               \
    } while (0)

static uint64_t rng = 88172645463325252ull;
static double urand(void)
{
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (double)(rng >> 11) / 9007199254740992.0 * 2.0 - 1.0;
}
static double *vec(size_t n, int ones)
{
    double *x = (double *)malloc(sizeof(double) * (n ? n : 1));
    for (size_t i = 0; i < n; ++i) x[i] = ones ? 1.0 : urand();
    return x;
}
/* weights: per level l, rank p bases of length s_l (2D: pairs [x | y]) */
static double *weights(int64_t r, int L, int64_t p, int two_d, int uniform)
{
    int64_t len = 0;
    for (int l = 1; l < L; ++l) len += p * (two_d ? 2 : 1) * (r << (l - 1));
    double *w = (double *)malloc(sizeof(double) * (len ? len : 1));
    int64_t o = 0;
    for (int l = 1; l < L; ++l) {
        const int64_t s = r << (l - 1);
        for (int64_t b = 0; b < p * (two_d ? 2 : 1); ++b)
            for (int64_t j = 0; j < s; ++j) w[o++] = uniform ? 1.0 / s : urand() / sqrt((double)s);
    }
    return w;
}

static void case_1d(int64_t n, int64_t r, int causal, int64_t p, int norm)
{
    const int64_t d = 8, S = 2;
    const int L = fmao_num_levels(n / r);
    double *q = vec(S * n * d, 0), *k = vec(S * n * d, 0), *v1 = vec(S * n * d, 1), *v = vec(S * n * d, 0);
    double *wk = weights(r, L, p, 0, 0), *wv1 = weights(r, L, p, 0, 1);
    double *o = vec(S * n * d, 0);
    int64_t *cnt = (int64_t *)malloc(sizeof(int64_t) * S * n);
    CHECK(fmao_forward_1d(q, k, v1, S, n, d, r, causal, p, wk, wv1, NULL, 0, 0.125, norm, o, cnt) == 0);
    /* weights sum to one (a clipped last group of a ragged sequence sums
       fewer than s weights of 1/s, so only whole groups are checked) */
    const int whole = (n / r & (n / r - 1)) == 0;
    if (norm == 0 && whole)
        for (int64_t i = 0; i < S * n * d; ++i) CHECK(fabs(o[i] - 1.0) < 1e-12);
    /* causality: perturb tokens after t, rows <= t unchanged */
    double *o2 = vec(S * n * d, 0);
    CHECK(fmao_forward_1d(q, k, v, S, n, d, r, causal, p, wk, wk, NULL, 0, 0.125, norm, o, cnt) == 0);
    if (causal) {
        const int64_t t = n / 2 + 3;
        double *k2 = vec(S * n * d, 0);
        memcpy(k2, k, sizeof(double) * (size_t)(S * n * d));
        for (int64_t i = t + 1; i < n; ++i) k2[i * d] += 5.0;
        CHECK(fmao_forward_1d(q, k2, v, S, n, d, r, causal, p, wk, wk, NULL, 0, 0.125, norm, o2, cnt) == 0);
        for (int64_t i = 0; i < (t + 1) * d; ++i) CHECK(o2[i] == o[i]);
        free(k2);
    }
    /* FMA-linear (bidirectional, rank 1, joint) */
    if (!causal && p == 1 && norm == 0)
        CHECK(fmao_forward_1d(q, k, v, S, n, d, r, 0, 1, wk, wk, wk, 0, 0.125, 0, o2, cnt) == 0);
    /* coarsening, lists */
    const int64_t R = p * fmao_coarse_rows_1d(n, r);
    double *cb = vec(R * d, 0);
    if (L > 1) CHECK(fmao_coarsen_1d(k, n, d, r, p, wk, cb) == 0);
    const int64_t nb = n / r;
    int32_t *lists = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nb * (L > 1 ? L - 1 : 1) * 3));
    int64_t *lo = (int64_t *)malloc(sizeof(int64_t) * nb), *hi = (int64_t *)malloc(sizeof(int64_t) * nb);
    CHECK(fmao_lists_1d(n, r, 3, lists, lo, hi) == 0);
    /* backward */
    double *dq = vec(S * n * d, 0), *dk = vec(S * n * d, 0), *dv = vec(S * n * d, 0);
    int64_t wl = 0;
    for (int l = 1; l < L; ++l) wl += p * (r << (l - 1));
    double *dpk = vec(S * (wl ? wl : 1), 0), *dpv = vec(S * (wl ? wl : 1), 0);
    CHECK(fmao_backward_1d(q, k, v, S, n, d, r, causal, p, wk, wk, 0, 0.125, norm, v1, dq, dk, dv, dpk, dpv) == 0);
    for (int64_t i = 0; i < S * n * d; ++i) CHECK(isfinite(dq[i]) && isfinite(dk[i]) && isfinite(dv[i]));
    free(q), free(k), free(v1), free(v), free(wk), free(wv1), free(o), free(o2), free(cnt), free(cb);
    free(lists), free(lo), free(hi), free(dq), free(dk), free(dv), free(dpk), free(dpv);
}

static void case_2d(int64_t W, int64_t r, int64_t p, int norm)
{
    const int64_t d = 4, S = 1, n = W * W;
    const int L = fmao_num_levels(W / r);
    double *q = vec(S * n * d, 0), *k = vec(S * n * d, 0), *v1 = vec(S * n * d, 1), *v = vec(S * n * d, 0);
    double *wk = weights(r, L, p, 1, 0), *wv1 = weights(r, L, p, 1, 1);
    double *o = vec(S * n * d, 0);
    int64_t *cnt = (int64_t *)malloc(sizeof(int64_t) * S * n);
    CHECK(fmao_forward_2d(q, k, v1, S, W, d, r, p, wk, wv1, NULL, 0, 0.5, norm, o, cnt) == 0);
    const int whole = (W / r & (W / r - 1)) == 0;
    if (norm == 0 && whole)
        for (int64_t i = 0; i < S * n * d; ++i) CHECK(fabs(o[i] - 1.0) < 1e-12);
    if (p == 1 && norm == 0) CHECK(fmao_forward_2d(q, k, v, S, W, d, r, 1, wk, wk, wk, 0, 0.5, 0, o, cnt) == 0);
    const int64_t R = p * fmao_coarse_rows_2d(W, r);
    double *cb = vec(R * d, 0);
    if (L > 1) CHECK(fmao_coarsen_2d(k, W, d, r, p, wk, cb) == 0);
    const int64_t nbx = W / r;
    int32_t *lists = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nbx * nbx * (L > 1 ? L - 1 : 1) * 27));
    CHECK(fmao_lists_2d(W, r, 27, lists) == 0);
    double *dq = vec(S * n * d, 0), *dk = vec(S * n * d, 0), *dv = vec(S * n * d, 0);
    int64_t wl = 0;
    for (int l = 1; l < L; ++l) wl += p * 2 * (r << (l - 1));
    double *dpk = vec(S * (wl ? wl : 1), 0), *dpv = vec(S * (wl ? wl : 1), 0);
    CHECK(fmao_backward_2d(q, k, v, S, W, d, r, p, wk, wk, 0, 0.5, norm, v1, dq, dk, dv, dpk, dpv) == 0);
    free(q), free(k), free(v1), free(v), free(wk), free(wv1), free(o), free(cnt), free(cb), free(lists);
    free(dq), free(dk), free(dv), free(dpk), free(dpv);
}

int main(void)
{
    for (int causal = 0; causal < 2; ++causal)
        for (int norm = 0; norm < 2; ++norm) {
            case_1d(64, 8, causal, 1, norm);
            case_1d(8 * 11, 8, causal, 1, norm);     /* n / r not a power of two */
            case_1d(256, 16, causal, 3, norm);
            case_1d(16, 16, causal, 1, norm);        /* one block */
            case_1d(32, 16, causal, 2, norm);        /* two blocks */
        }
    for (int norm = 0; norm < 2; ++norm) {
        case_2d(16, 2, 1, norm);
        case_2d(12, 2, 1, norm);                     /* W / r not a power of two */
        case_2d(16, 4, 2, norm);
        case_2d(4, 4, 1, norm);
    }
    /* bad arguments are rejected, not read */
    double x = 0.0, y = 0.0;
    int64_t c = 0;
    CHECK(fmao_forward_1d(NULL, &x, &x, 1, 8, 1, 4, 0, 1, NULL, NULL, NULL, 0, 1.0, 0, &y, &c) != 0);
    CHECK(fmao_forward_1d(&x, &x, &x, 1, 9, 1, 4, 0, 1, NULL, NULL, NULL, 0, 1.0, 0, &y, &c) != 0);
    CHECK(fmao_forward_2d(&x, &x, &x, 1, 6, 1, 4, 1, NULL, NULL, NULL, 0, 1.0, 0, &y, &c) != 0);
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("oracle checks passed\n");
    return 0;
}
