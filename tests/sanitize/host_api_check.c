/* Host-side checks of the C ABI under AddressSanitizer / UBSan (test
 * infrastructure).  Built against a host-only, sanitizer-instrumented build
 * of the library (no device code), so it exercises plan construction,
 * sizing, the plan-parameter export and every validation path -- and never
 * reaches a launch: each call given device pointers is built to fail
 * validation first (fake addresses are never dereferenced). */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "fma.h"

static int failures = 0;
#define CHECK(c)                                                                   \
    do {                                                                           \
        if (!(c)) {                                                                \
            fprintf(stderr, "FAIL line %d: %s (%s)\n", __LINE__, #c, fma_last_error()); \
            ++failures;                                                            \
        }                                                                          \
    } while (0)

static fma_desc_t desc(int ndim, int B, int H, long long n, int side, int r, int causal, int dtype, int rank,
                       int norm, int linear)
{
    fma_desc_t d;
    memset(&d, 0, sizeof(d));
    d.struct_size = (int32_t)sizeof(fma_desc_t);
    d.ndim = ndim;
    d.batch = B;
    d.heads = H;
    d.seq_len = n;
    d.side = side;
    d.head_dim = 64;
    d.block = r;
    d.num_levels = -1;
    d.causal = causal;
    d.dtype = dtype;
    d.weights_per_head = 1;
    d.rank = rank;
    d.norm = norm;
    d.query_downsample = linear;
    return d;
}

/* A valid plan: every query, then validation failures of every entry point. */
static void exercise(const fma_desc_t *d)
{
    fma_plan_t p = NULL;
    if (fma_plan(d, &p) != FMA_OK) return;   /* unsupported shapes are fine here */
    size_t ws = 0, bws = 0;
    int64_t wl = 0, rows = 0;
    int32_t L = 0, cnt = 0;
    CHECK(fma_workspace_size(p, &ws) == FMA_OK);
    CHECK(fma_backward_workspace_size(p, &bws) == FMA_OK);
    CHECK(fma_weights_len(p, &wl) == FMA_OK);
    CHECK(fma_coarse_rows(p, &rows) == FMA_OK);
    CHECK(fma_num_levels(p, &L) == FMA_OK);
    CHECK(bws >= ws);
    int64_t small[4];
    CHECK(fma_plan_params(p, small, 4, &cnt) == FMA_ERR_WORKSPACE && cnt > 4);
    int64_t *params = (int64_t *)malloc(sizeof(int64_t) * (size_t)cnt);   /* exact size */
    int32_t cnt2 = 0;
    CHECK(fma_plan_params(p, params, cnt, &cnt2) == FMA_OK && cnt2 == cnt);
    CHECK(params[7] == rows && params[17] == wl);
    free(params);

    /* fake, aligned device addresses far apart (never dereferenced) */
    void *q = (void *)(uintptr_t)0x100000000ull, *k = (void *)(uintptr_t)0x200000000ull;
    void *v = (void *)(uintptr_t)0x300000000ull, *o = (void *)(uintptr_t)0x400000000ull;
    void *w = (void *)(uintptr_t)0x500000000ull;
    const float *wk = (const float *)(uintptr_t)0x600000000ull, *wv = (const float *)(uintptr_t)0x700000000ull;
    const int empty = d->batch == 0 || d->heads == 0 || d->seq_len == 0;
    if (!empty) {
        const int fwd1 = d->ndim == 1 && !d->query_downsample;
        fma_status_t (*fwd)(fma_plan_t, const void *, const void *, const void *, const float *, const float *,
                            void *, void *, size_t, void *) = d->ndim == 1 ? fma_forward_1d : fma_forward_2d;
        if (!d->query_downsample) {
            CHECK(fwd(p, NULL, k, v, wk, wv, o, w, ws, NULL) == FMA_ERR_NULL);
            CHECK(fwd(p, (char *)q + 2, k, v, wk, wv, o, w, ws, NULL) == FMA_ERR_ALIGN);
            CHECK(fwd(p, q, k, v, wk, wv, q, w, ws, NULL) == FMA_ERR_ARG);   /* out aliases q */
            if (ws > 0) {
                CHECK(fwd(p, q, k, v, wk, wv, o, w, ws - 1, NULL) == FMA_ERR_WORKSPACE);
                CHECK(fwd(p, q, k, v, wk, wv, o, NULL, ws, NULL) == FMA_ERR_WORKSPACE);
                CHECK(fwd(p, q, k, v, NULL, wv, o, w, ws, NULL) == FMA_ERR_NULL);
            }
            /* the other dimension's entry point */
            CHECK((fwd1 ? fma_forward_2d : fma_forward_1d)(p, q, k, v, wk, wv, o, w, ws, NULL) == FMA_ERR_SHAPE);
            CHECK(fma_attend(p, q, k, v, w, ws, NULL, NULL) == FMA_ERR_NULL);
            if (ws > 0) CHECK(fma_coarsen(p, k, v, wk, wv, w, ws - 1, NULL) == FMA_ERR_WORKSPACE);
            CHECK(fma_forward_linear(p, q, k, v, wk, wk, wv, o, w, ws, NULL) == FMA_ERR_ARG);
            if (ws > ((size_t)32 << 20))
                CHECK(fma_forward_static(p, q, k, v, wk, wv, o, NULL) == FMA_ERR_WORKSPACE);
            else
                CHECK(fma_forward_static(p, NULL, k, v, wk, wv, o, NULL) == FMA_ERR_NULL);
        } else {
            CHECK(fwd(p, q, k, v, wk, wv, o, w, ws, NULL) == FMA_ERR_ARG);   /* FMA-linear plan */
            if (wl > 0) CHECK(fma_forward_linear(p, q, k, v, NULL, wk, wv, o, w, ws, NULL) == FMA_ERR_NULL);
            CHECK(fma_forward_static(p, q, k, v, wk, wv, o, NULL) == FMA_ERR_ARG);
        }
        {
            void *dq = (void *)(uintptr_t)0x800000000ull, *dk = (void *)(uintptr_t)0x900000000ull;
            void *dv = (void *)(uintptr_t)0xa00000000ull;
            float *dwk = (float *)(uintptr_t)0xb00000000ull, *dwv = (float *)(uintptr_t)0xc00000000ull;
            float *dwq = (float *)(uintptr_t)0xd00000000ull;
            if (!d->query_downsample) {
                CHECK(fma_backward(p, q, k, v, wk, wv, o, o, dq, dk, dv, dwk, dwv, w, bws - 1, NULL) ==
                      FMA_ERR_WORKSPACE);
                CHECK(fma_backward(p, q, k, v, wk, wv, o, o, dq, dq, dv, dwk, dwv, w, bws, NULL) == FMA_ERR_ARG);
                CHECK(fma_backward_linear(p, q, k, v, wk, wv, wk, o, o, dq, dk, dv, dwk, dwv, dwq, w, bws, NULL) ==
                      FMA_ERR_ARG);
            } else {
                CHECK(fma_backward(p, q, k, v, wk, wv, o, o, dq, dk, dv, dwk, dwv, w, bws, NULL) == FMA_ERR_ARG);
                CHECK(fma_backward_linear(p, q, k, v, wk, wv, wk, o, o, dq, dk, dv, dwk, dwv, dwq, w, bws - 1,
                                          NULL) == FMA_ERR_WORKSPACE);
                CHECK(fma_backward_linear(p, q, k, v, wk, wv, wk, o, o, dq, dq, dv, dwk, dwv, dwq, w, bws, NULL) ==
                      FMA_ERR_ARG);
                if (wl > 0)
                    CHECK(fma_backward_linear(p, q, k, v, wk, wv, NULL, o, o, dq, dk, dv, dwk, dwv, dwq, w, bws,
                                              NULL) == FMA_ERR_NULL);
            }
        }
    }
    CHECK(fma_destroy(p) == FMA_OK);
}

int main(void)
{
    /* valid plans across the supported space */
    static const int rs1[] = {64, 128, 192, 256};
    static const long long mult[] = {1, 2, 3, 4, 7, 8, 16, 37, 64, 512};
    for (int ri = 0; ri < 4; ++ri)
        for (int mi = 0; mi < 10; ++mi)
            for (int causal = 0; causal < 2; ++causal)
                for (int rank = 1; rank <= 5; rank += 2)
                    for (int norm = 0; norm < 2; ++norm)
                        for (int dt = 0; dt < 2; ++dt) {
                            fma_desc_t d = desc(1, 2, 3, rs1[ri] * mult[mi], 0, rs1[ri], causal, dt, rank, norm, 0);
                            exercise(&d);
                        }
    for (int mi = 0; mi < 10; ++mi) {
        fma_desc_t d = desc(1, 2, 3, 128 * mult[mi], 0, 128, 0, 1, 1, 0, 1);
        exercise(&d);
    }
    static const int sides[] = {8, 16, 24, 32, 40, 64, 80, 96, 128, 256};
    for (int si = 0; si < 10; ++si)
        for (int r = 8; r <= 16; r += 8)
            for (int rank = 1; rank <= 4; rank += 3)
                for (int norm = 0; norm < 2; ++norm)
                    for (int dt = 0; dt < 2; ++dt) {
                        if (sides[si] % r) continue;
                        fma_desc_t d = desc(2, 1, 2, (long long)sides[si] * sides[si], sides[si], r, 0, dt, rank,
                                            norm, 0);
                        exercise(&d);
                        d.query_downsample = 1;
                        d.rank = 1;
                        d.norm = 0;
                        exercise(&d);
                    }
    /* the empty problem */
    {
        fma_desc_t d = desc(1, 0, 4, 1024, 0, 64, 0, 1, 1, 0, 0);
        exercise(&d);
    }
    /* invalid descriptors, each with its documented status and a message */
    {
        fma_plan_t p = NULL;
        fma_desc_t d = desc(1, 1, 1, 1000, 0, 64, 0, 1, 1, 0, 0);
        CHECK(fma_plan(&d, &p) == FMA_ERR_SHAPE && p == NULL && fma_last_error()[0]);
        d = desc(1, 1, 1, 1024, 0, 64, 0, 1, 1, 0, 0);
        d.head_dim = 96;   /* 32, 64 and 128 are built */
        CHECK(fma_plan(&d, &p) == FMA_ERR_UNSUPPORTED && p == NULL);
        d = desc(1, 1, 1, 1024, 0, 64, 0, 7, 1, 0, 0);
        CHECK(fma_plan(&d, &p) == FMA_ERR_ARG);
        d = desc(1, 1, 1, 1024, 0, 64, 0, 1, -1, 0, 0);
        CHECK(fma_plan(&d, &p) == FMA_ERR_ARG);
        d = desc(2, 1, 1, 64 * 64, 64, 8, 1, 1, 1, 0, 0);
        CHECK(fma_plan(&d, &p) == FMA_ERR_UNSUPPORTED);
        d = desc(2, 1, 1, 64 * 60, 64, 8, 0, 1, 1, 0, 0);
        CHECK(fma_plan(&d, &p) == FMA_ERR_SHAPE);
        d = desc(1, 1, 1, 1024, 0, 64, 1, 1, 1, 0, 1);
        CHECK(fma_plan(&d, &p) == FMA_ERR_UNSUPPORTED);
        d = desc(1, 1, 1, 1024, 0, 64, 0, 1, 1, 0, 0);
        d.num_levels = 3;
        CHECK(fma_plan(&d, &p) == FMA_ERR_SHAPE);
        d.struct_size = 12;
        CHECK(fma_plan(&d, &p) == FMA_ERR_ARG);
        CHECK(fma_plan(NULL, &p) == FMA_ERR_NULL);
        CHECK(fma_destroy(NULL) == FMA_OK);
        /* descriptors without the rank / query_downsample fields */
        d = desc(1, 1, 1, 1024, 0, 64, 0, 1, 1, 0, 0);
        d.struct_size = (int32_t)offsetof(fma_desc_t, rank);
        CHECK(fma_plan(&d, &p) == FMA_OK);
        CHECK(fma_destroy(p) == FMA_OK);
        d.struct_size = (int32_t)offsetof(fma_desc_t, query_downsample);
        CHECK(fma_plan(&d, &p) == FMA_OK);
        CHECK(fma_destroy(p) == FMA_OK);
    }
    /* the bench export's validation */
    {
        void *a = (void *)(uintptr_t)0x100000000ull, *b = (void *)(uintptr_t)0x200000000ull;
        CHECK(fma_stream_reference(NULL, 1024, b, 1 << 20, 64, NULL) == FMA_ERR_NULL);
        CHECK(fma_stream_reference(a, 1024, b, 1 << 20, 63, NULL) == FMA_ERR_ARG);
        CHECK(fma_stream_reference(a, 1 << 20, b, 16, 64, NULL) == FMA_ERR_WORKSPACE);
        CHECK(fma_stream_reference(a, 1 << 20, (char *)a + 4096, 1 << 20, 64, NULL) == FMA_ERR_ARG);
    }
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("host api checks passed\n");
    return 0;
}
