/*
 * Drives the fp64 oracle (oracle/kvr_ref.c) under AddressSanitizer and
 * UndefinedBehaviorSanitizer: tiny shapes, every entry point, several thread
 * counts, and canary rows around every cache range the oracle must not read
 * or write.  Exit status 0 when every check holds; the sanitizers abort the
 * process on the first finding.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int kvr_ref_prefill(int n_q_heads, int n_kv_heads, int head_dim, double scale, const double *Q, const double *K,
                    const double *V, int64_t L, const int64_t *rows, int64_t n_rows, double *out, double *lse,
                    int nthreads);
int kvr_ref_continue(int n_q_heads, int n_kv_heads, int head_dim, double scale, const double *Qs, const double *Ks,
                     const double *Vs, int64_t S, const double *kcache, const double *vcache, int64_t capacity,
                     int64_t L_prefix, int64_t k_lo, int64_t k_hi, const int64_t *rows, int64_t n_rows, double *out,
                     double *lse, int nthreads);
int kvr_ref_cache_append(int n_kv_heads, int head_dim, const double *Ks, const double *Vs, int64_t S,
                         double *kcache, double *vcache, int64_t capacity, int64_t L_cur);

static uint64_t rng = 0x9e3779b97f4a7c15ull;
static double urand(void) {
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (double)(rng >> 11) / 9007199254740992.0 * 2.0 - 1.0;
}
static double *alloc_fill(size_t n) {
    double *p = (double *)malloc((n ? n : 1) * sizeof(double));
    for (size_t i = 0; i < n; ++i) p[i] = urand() * 2.0;
    return p;
}

static int fails = 0;
#define CHECK(c, ...)                      \
    do {                                   \
        if (!(c)) {                        \
            fprintf(stderr, __VA_ARGS__);  \
            fputc('\n', stderr);           \
            ++fails;                       \
        }                                  \
    } while (0)

static void one_shape(int Hq, int Hkv, int d, int64_t N, int nthreads) {
    const double scale = 1.0 / sqrt((double)d);
    const int64_t cap = N + 3;   /* rows N.. are canaries */
    double *Q = alloc_fill((size_t)N * Hq * d), *K = alloc_fill((size_t)N * Hkv * d);
    double *V = alloc_fill((size_t)N * Hkv * d);
    double *full = (double *)malloc((size_t)(N ? N : 1) * Hq * d * sizeof(double));
    double *lse = (double *)malloc((size_t)(N ? N : 1) * Hq * sizeof(double));
    CHECK(kvr_ref_prefill(Hq, Hkv, d, scale, Q, K, V, N, NULL, N, full, lse, nthreads) == 0, "prefill failed");

    /* a row subset, in list order */
    if (N >= 2) {
        const int64_t rows[2] = {N - 1, 0};
        double *sub = (double *)malloc((size_t)2 * Hq * d * sizeof(double));
        double *sl = (double *)malloc((size_t)2 * Hq * sizeof(double));
        CHECK(kvr_ref_prefill(Hq, Hkv, d, scale, Q, K, V, N, rows, 2, sub, sl, nthreads) == 0, "prefill rows failed");
        CHECK(memcmp(sub, full + (size_t)(N - 1) * Hq * d, (size_t)Hq * d * sizeof(double)) == 0, "row subset differs");
        CHECK(memcmp(sub + (size_t)Hq * d, full, (size_t)Hq * d * sizeof(double)) == 0, "row subset differs");
        free(sub);
        free(sl);
    }

    /* caches with NaN canaries past the written rows */
    double *kc = (double *)malloc((size_t)Hkv * cap * d * sizeof(double));
    double *vc = (double *)malloc((size_t)Hkv * cap * d * sizeof(double));
    for (size_t i = 0; i < (size_t)Hkv * cap * d; ++i) kc[i] = vc[i] = NAN;
    const int64_t cuts[4] = {0, 1, N / 2, N > 0 ? N - 1 : 0};
    for (int ci = 0; ci < 4; ++ci) {
        const int64_t Lp = cuts[ci] <= N ? cuts[ci] : N, S = N - Lp;
        for (size_t i = 0; i < (size_t)Hkv * cap * d; ++i) kc[i] = vc[i] = NAN;
        CHECK(kvr_ref_cache_append(Hkv, d, K, V, Lp, kc, vc, cap, 0) == 0, "append failed");
        double *out = (double *)malloc((size_t)(S ? S : 1) * Hq * d * sizeof(double));
        double *ls = (double *)malloc((size_t)(S ? S : 1) * Hq * sizeof(double));
        CHECK(kvr_ref_continue(Hq, Hkv, d, scale, Q + (size_t)Lp * Hq * d, K + (size_t)Lp * Hkv * d,
                               V + (size_t)Lp * Hkv * d, S, kc, vc, cap, Lp, 0, Lp + S, NULL, S, out, ls,
                               nthreads) == 0,
              "continue failed");
        double worst = 0.0;
        for (size_t i = 0; i < (size_t)S * Hq * d; ++i) {
            const double e = fabs(out[i] - full[(size_t)Lp * Hq * d + i]);
            if (!(e <= worst)) worst = e;   /* NaN propagates into worst */
        }
        CHECK(worst <= 1e-12, "continue vs prefill rows: %g (N=%ld Lp=%ld)", worst, (long)N, (long)Lp);
        /* an empty key range: out 0, lse -inf */
        if (S > 0) {
            CHECK(kvr_ref_continue(Hq, Hkv, d, scale, Q + (size_t)Lp * Hq * d, K + (size_t)Lp * Hkv * d,
                                   V + (size_t)Lp * Hkv * d, S, kc, vc, cap, Lp, 0, 0, NULL, S, out, ls,
                                   nthreads) == 0,
                  "empty-range continue failed");
            CHECK(out[0] == 0.0 && isinf(ls[0]) && ls[0] < 0, "empty key range");
        }
        /* the rest of the cache, appended after the prefix: rows [0, N) equal K/V, canaries stay */
        CHECK(kvr_ref_cache_append(Hkv, d, K + (size_t)Lp * Hkv * d, V + (size_t)Lp * Hkv * d, S, kc, vc, cap,
                                   Lp) == 0,
              "second append failed");
        for (int g = 0; g < Hkv; ++g)
            for (int64_t r = 0; r < cap; ++r)
                for (int c = 0; c < d; ++c) {
                    const double got = kc[((size_t)g * cap + r) * d + c];
                    if (r < N) CHECK(got == K[((size_t)r * Hkv + g) * d + c], "cache row %ld", (long)r);
                    else CHECK(isnan(got), "canary row %ld overwritten", (long)r);
                }
        free(out);
        free(ls);
    }
    CHECK(kvr_ref_cache_append(Hkv, d, K, V, 4, kc, vc, cap, cap - 3) == 1, "append past capacity accepted");
    CHECK(kvr_ref_continue(Hq, Hkv, d, scale, Q, K, V, 0, kc, vc, cap, cap + 1, 0, 0, NULL, 0, full, lse,
                           nthreads) == 1,
          "prefix past capacity accepted");
    free(Q); free(K); free(V); free(full); free(lse); free(kc); free(vc);
}

int main(void) {
    const int shapes[][3] = {{2, 1, 8}, {4, 2, 16}, {3, 3, 4}, {8, 2, 8}};
    const int64_t lens[] = {1, 2, 17, 40};
    const int threads[] = {1, 3, 8};
    for (int s = 0; s < 4; ++s)
        for (int n = 0; n < 4; ++n)
            for (int t = 0; t < 3; ++t) one_shape(shapes[s][0], shapes[s][1], shapes[s][2], lens[n], threads[t]);
    if (fails) {
        fprintf(stderr, "%d checks failed\n", fails);
        return 1;
    }
    printf("oracle driver: all checks passed\n");
    return 0;
}
