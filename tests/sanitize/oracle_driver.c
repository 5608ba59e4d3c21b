/* oracle_driver.c -- runs the CPU oracle (oracle/roi_oracle.c) over edge
 * shapes under the host compiler's address and undefined-behaviour
 * sanitizers: n = m, m = 32 and 64 (its largest group), groups whose
 * log(1 - mu) is floored, arrays of zero and one group, odd group counts for
 * the 2:4 metadata, the categorical sampler at its largest candidate count,
 * the threaded entry points, and rejected arguments.  Each run also checks
 * what it can about its outputs (n kept per group, sum S = n). */
#include "roi_oracle.h"

#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static int failures = 0;

#define EXPECT(cond, ...)                                                                      \
    do {                                                                                       \
        if (!(cond)) {                                                                         \
            printf("FAIL line %d: ", __LINE__);                                                \
            printf(__VA_ARGS__);                                                               \
            printf("\n");                                                                      \
            ++failures;                                                                        \
        }                                                                                      \
    } while (0)

static uint32_t rng_state = 12345u;
static double unit(void) /* xorshift32 in (0, 1) */
{
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 17;
    rng_state ^= rng_state << 5;
    return ((double)rng_state + 0.5) / 4294967296.0;
}
static double normal(void) { return sqrt(-2.0 * log(unit())) * cos(6.283185307179586 * unit()); }
static uint16_t bf16(double x)
{
    float f = (float)x;
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

/* forward and backward over `groups` groups of m; spike: one logit per group
 * raised by `spike` (its 1 - mu falls below FLT_MIN when spike >> tau) */
static void run(int n, int m, int64_t groups, float tau, float lambda, double spike, int threads)
{
    const int64_t numel = groups * m;
    size_t cnt = numel ? (size_t)numel : 1;
    uint16_t* W = malloc(cnt * 2);
    uint16_t* G = malloc(cnt * 2);
    float* L = malloc(cnt * 4);
    uint16_t* Wm = malloc(cnt * 2);
    double* S = malloc(cnt * 8);
    double* d = malloc(cnt * 8);
    uint8_t* idx = malloc((size_t)(groups ? groups : 1) * (size_t)n);
    for (int64_t i = 0; i < numel; ++i) {
        W[i] = bf16(0.02 * normal());
        G[i] = bf16(normal());
        L[i] = (float)normal() + ((i % m) == (i / m) % m ? (float)spike : 0.0f);
    }
    const uint64_t off = 4ull << 32;
    int rc = threads > 1
                 ? roi_oracle_fwd_mt(W, L, numel, n, m, tau, lambda, 7, 3, off, Wm, S, idx, threads)
                 : roi_oracle_fwd(W, L, numel, n, m, tau, lambda, 7, 3, off, Wm, S, idx);
    EXPECT(rc == 0, "fwd %d:%d groups %lld rc %d", n, m, (long long)groups, rc);
    for (int64_t q = 0; q < groups; ++q) {
        int kept = 0;
        double s = 0.0;
        for (int j = 0; j < m; ++j) {
            kept += Wm[q * m + j] == W[q * m + j] && W[q * m + j] != 0;
            s += S[q * m + j];
        }
        uint8_t seen[64] = {0};
        for (int r = 0; r < n; ++r) {
            EXPECT(idx[q * n + r] < m && !seen[idx[q * n + r]], "index %d", idx[q * n + r]);
            if (idx[q * n + r] < m) seen[idx[q * n + r]] = 1;
        }
        EXPECT(kept <= n, "group %lld keeps %d > %d", (long long)q, kept, n);
        EXPECT(fabs(s - n) < 1e-9 * n, "group %lld: sum S = %.17g, n = %d", (long long)q, s, n);
    }
    rc = threads > 1
             ? roi_oracle_bwd_mt(G, W, L, numel, n, m, tau, lambda, 7, 3, off, d, threads)
             : roi_oracle_bwd(G, W, L, numel, n, m, tau, lambda, 7, 3, off, d);
    EXPECT(rc == 0, "bwd %d:%d rc %d", n, m, rc);
    for (int64_t i = 0; i < numel; ++i) EXPECT(isfinite(d[i]), "non-finite gradient at %lld", (long long)i);
    free(W); free(G); free(L); free(Wm); free(S); free(d); free(idx);
}

int main(void)
{
    /* patterns: n = m, wide groups, the largest group, one and zero groups */
    run(4, 4, 33, 1.0f, 1.0f, 0.0, 1);
    run(2, 4, 1, 0.5f, 1.0f, 0.0, 1);
    run(2, 4, 0, 0.5f, 1.0f, 0.0, 1);
    run(8, 8, 17, 0.3f, 0.7f, 0.0, 1);
    run(16, 32, 9, 1.0f, 1.0f, 0.0, 1);
    run(32, 32, 5, 0.9f, 1.0f, 0.0, 1);
    run(31, 32, 3, 1.0f, 2.0f, 0.0, 1);
    run(40, 64, 2, 1.0f, 1.0f, 0.0, 1);
    /* floored groups: one key 100 (and 250) above the rest */
    run(2, 4, 64, 1.0f, 1.0f, 100.0, 1);
    run(3, 4, 64, 0.5f, 1.0f, 100.0, 1);
    run(3, 8, 16, 1.0f, 1.0f, 250.0, 1);
    run(8, 16, 8, 1.0f, 1.0f, 150.0, 1);
    /* the threaded entry points, more threads than groups */
    run(2, 4, 1001, 1.0f, 1.0f, 0.0, 7);
    run(4, 8, 3, 0.5f, 1.0f, 100.0, 16);
    run(2, 4, 0, 1.0f, 1.0f, 0.0, 4);

    /* relaxation on explicit keys, and many groups at once */
    {
        double k[64], sb[64], dk[64], S[64];
        for (int j = 0; j < 64; ++j) {
            k[j] = normal();
            sb[j] = normal();
        }
        EXPECT(oracle_relax_fwd(k, 64, 64, 1.0, S) == 0, "relax_fwd 64:64");
        EXPECT(oracle_relax_bwd(k, 64, 1, 0.2, sb, dk) == 0, "relax_bwd 1:64");
        EXPECT(oracle_relax_bwd_groups(k, 2, 32, 16, 1.0, sb, dk, 5) == 0, "relax_bwd_groups");
        EXPECT(oracle_relax_bwd_groups(k, 0, 32, 16, 1.0, sb, dk, 5) == 0, "relax_bwd_groups 0");
        uint8_t order[64], hard[64];
        float kf[64];
        for (int j = 0; j < 64; ++j) kf[j] = (float)(j % 3);
        EXPECT(oracle_topn(kf, 64, 64, order, hard) == 0, "topn 64:64");
        EXPECT(order[0] == 2 && order[63] == 63, "topn ties to the lower index");
    }

    /* export with a partial last metadata word, and the categorical sampler */
    {
        const int groups = 13, m = 4;
        float L[13 * 4];
        uint16_t W[13 * 4], Wm[13 * 4], vals[13 * 2];
        uint8_t idx[13 * 2];
        uint32_t meta[2];
        for (int i = 0; i < groups * m; ++i) {
            L[i] = (float)normal();
            W[i] = bf16(normal());
        }
        EXPECT(oracle_export(L, W, groups * m, 2, m, Wm, vals, idx, meta) == 0, "export 2:4");
        EXPECT(oracle_export(L, W, 0, 2, m, Wm, vals, idx, meta) == 0, "export empty");
        EXPECT(oracle_export(L, W, groups * m, 3, m, Wm, vals, idx, meta) != 0,
               "metadata only for 2:4");
        EXPECT(oracle_export(L, W, 8 * 5, 5, 8, Wm, vals, idx, NULL) == 0, "export 5:8");
    }
    {
        uint32_t masks[70];
        EXPECT(oracle_cat_candidates(4, 8, masks) == 70, "70 candidates at 4:8");
        EXPECT(oracle_cat_candidates(8, 8, masks) == 1, "one candidate at 8:8");
        const int groups = 5, m = 8, n = 4, C = 70;
        float A[5 * 70];
        uint16_t W[5 * 8], G[5 * 8], Wm[5 * 8];
        double S[5 * 8], dA[5 * 70];
        uint8_t choice[5];
        for (int i = 0; i < groups * C; ++i) A[i] = (float)normal();
        for (int i = 0; i < groups * m; ++i) {
            W[i] = bf16(normal());
            G[i] = bf16(normal());
        }
        EXPECT(oracle_cat_fwd(W, A, groups, n, m, 0.5f, 1.0f, 1, 2, 1ull << 40, Wm, S, choice) == 0,
               "cat fwd 4:8");
        EXPECT(oracle_cat_bwd(G, W, A, groups, n, m, 0.5f, 1.0f, 1, 2, 1ull << 40, dA) == 0,
               "cat bwd 4:8");
        for (int q = 0; q < groups; ++q) {
            double s = 0.0;
            for (int j = 0; j < m; ++j) s += S[q * m + j];
            EXPECT(fabs(s - n) < 1e-9 * n && choice[q] < C, "cat group %d", q);
        }
        EXPECT(oracle_cat_fwd(W, A, 0, n, m, 0.5f, 1.0f, 1, 2, 0, Wm, S, choice) == 0, "cat empty");
    }

    /* rejected arguments */
    {
        uint16_t W[4] = {0}, Wm[4];
        float L[4] = {0};
        double S[4], k[4] = {0}, d[4];
        EXPECT(roi_oracle_fwd(W, L, 4, 5, 4, 1.0f, 1.0f, 0, 0, 0, Wm, S, NULL) != 0, "n > m");
        EXPECT(roi_oracle_fwd(W, L, 6, 2, 4, 1.0f, 1.0f, 0, 0, 0, Wm, S, NULL) != 0, "numel %% m");
        EXPECT(roi_oracle_fwd(W, L, 4, 2, 4, 0.0f, 1.0f, 0, 0, 0, Wm, S, NULL) != 0, "tau = 0");
        EXPECT(roi_oracle_fwd(W, L, 4, 2, 4, 1.0f, NAN, 0, 0, 0, Wm, S, NULL) != 0, "lambda NaN");
        EXPECT(oracle_relax_bwd(k, 65, 2, 1.0, k, d) != 0, "m = 65");
        EXPECT(oracle_relax_fwd(k, 4, 0, 1.0, S) != 0, "n = 0");
        uint32_t masks[70];
        EXPECT(oracle_cat_candidates(2, 9, masks) < 0, "m = 9");
        EXPECT(oracle_adamw(d, 4, 1e-3, 1.0, 0.9, 1e-8, 0.0, 1, L, L, L, d, d, d) != 0,
               "beta1 = 1");
    }
    if (failures) {
        printf("%d failures\n", failures);
        return 1;
    }
    printf("oracle ok\n");
    return 0;
}
