/*
 * roi_oracle.c -- plain, slow, scalar CPU oracle of the RoI
 * differentiable N:M mask sampler (arxiv 2608.23048, "Reservoir of Importance").
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may load this library.  It
 * shares no code, header, table or constant with the HIP library; the two
 * agree only because both follow the same written definitions below.
 *
 * What is computed, per group of m consecutive weights (§4.1: a mask keeps
 * exactly n of every m contiguous parameters):
 *
 *   1. noise      u_j ~ U(0,1) from a counter-based generator, g_j = -log(-log u_j)
 *                 (Appendix, Algorithm 1: Gumbel noise);
 *   2. keys       kappa_j = phi_j / lambda + g_j
 *                 (§3.2 / §4.2.2 key equation; §4.2.3: the Gumbel trick is
 *                 applied to the scaled logits phi / lambda);
 *   3. hard mask  the n largest keys, i.e. arg-top-n (§3.2 Gumbel-Top-K; the
 *                 straight-through variant of the appendix emits this mask in
 *                 the forward pass), so W_masked = W (.) hard (§4.1);
 *   4. relaxation alpha^(1) = kappa, mu^(k) = softmax(alpha^(k)/tau),
 *                 alpha^(k+1) = alpha^(k) + log(1 - mu^(k)),  S = sum_k mu^(k)
 *                 (§3.2 recursion, §4.2.2, Algorithm 1);
 *   5. backward   reverse-mode derivative of S with respect to phi, with the
 *                 upstream gradient of S equal to dL/dW_masked (.) W (the
 *                 straight-through estimator: backward through the relaxation).
 *
 * Readings of points the paper leaves open (each also listed in the design
 * notes):
 *   - u comes from Philox4x32-10 (Salmon et al., SC'11) keyed by the seed,
 *     with counter (element/4, step) and word element%4; u is the odd 23-bit
 *     grid point (2*(x>>9)+1) * 2^-24, never 0 or 1.
 *   - "log" in the noise is the deterministic fp32 logarithm oracle_log()
 *     below, so that the keys, and therefore the hard selection, are one
 *     well-defined fp32 value for every input.
 *   - keys are fp32: kappa = fl(fl(phi / lambda) + g).
 *   - ties between keys go to the lower index; the returned indices are in
 *     selection order (descending key).
 *   - the relaxation and its derivative run in fp64 from the fp32 keys;
 *     1 - mu_i is evaluated as sum_{j != i} mu_j (same value, no cancellation)
 *     and log(1 - mu) is floored at log(FLT_MIN) with zero derivative there.
 *   - pruned weights are +0.0 (bf16 bits 0x0000).
 */
#include "roi_oracle.h"

#include <float.h>
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_MAX_M 64

/* ------------------------------------------------------------------------- *
 * 1. Counter-based uniform source: Philox4x32-10 as published by Salmon,
 *    Moraes, Dror and Shaw ("Parallel random numbers: as easy as 1, 2, 3",
 *    SC'11).  Round: two 32x32->64 products of the even words with the two
 *    Philox multipliers, the high halves xor-ed with the odd words and the
 *    round key; the key advances by the two Weyl increments between rounds.
 * ------------------------------------------------------------------------- */
static const uint32_t PHILOX_MULT_A = 0xD2511F53u;
static const uint32_t PHILOX_MULT_B = 0xCD9E8D57u;
static const uint32_t WEYL_A = 0x9E3779B9u; /* golden ratio */
static const uint32_t WEYL_B = 0xBB67AE85u; /* sqrt(3) - 1 */

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += WEYL_A;
            k1 += WEYL_B;
        }
        uint64_t pa = (uint64_t)PHILOX_MULT_A * (uint64_t)c0;
        uint64_t pb = (uint64_t)PHILOX_MULT_B * (uint64_t)c2;
        uint32_t pa_hi = (uint32_t)(pa >> 32), pa_lo = (uint32_t)pa;
        uint32_t pb_hi = (uint32_t)(pb >> 32), pb_lo = (uint32_t)pb;
        uint32_t n0 = pb_hi ^ c1 ^ k0;
        uint32_t n1 = pb_lo;
        uint32_t n2 = pa_hi ^ c3 ^ k1;
        uint32_t n3 = pa_lo;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Word for global element `elem` at training step `step`. */
uint32_t oracle_philox_word(uint64_t seed, uint64_t step, uint64_t elem)
{
    uint64_t block = elem / 4u;
    uint32_t ctr[4] = {(uint32_t)block, (uint32_t)(block >> 32), (uint32_t)step,
                       (uint32_t)(step >> 32)};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    oracle_philox4x32_10(ctr, key, out);
    return out[elem % 4u];
}

/* u ~ U(0,1): the odd points of the 2^-24 grid, (2k+1) 2^-24 for the top 23
 * bits k of the word.  Exact in fp32; the extreme values are 2^-24 and
 * 1 - 2^-24. */
float oracle_uniform(uint32_t word)
{
    uint32_t k = word >> 9;
    double u = ((double)k * 2.0 + 1.0) / 16777216.0; /* exact */
    return (float)u;                                    /* exact */
}

/* ------------------------------------------------------------------------- *
 * 2. Deterministic fp32 natural logarithm (table-driven reduction in the
 *    manner of Tang, "Table-driven implementation of the logarithm function
 *    in IEEE floating-point arithmetic", ACM TOMS 1990), written from the
 *    mathematics:
 *      x = z 2^k with z in [0.703125, 1.40625)   (bit manipulation, exact)
 *      z lies in one of 128 cells: 76 cells of width 2^-8 below 1 and 52 of
 *      width 2^-7 from 1 up; cell i has centre c_i, inv_i = fl32(1/c_i) and
 *      lg_i = fl32(-ln inv_i), except the two cells touching 1, which use
 *      inv = 1 and lg = 0 so that r = z - 1 is exact there;
 *      r = fma(z, inv_i, -1)                      (|r| <= 2^-7)
 *      ln(1 + r) ~ r + r^2 (-1/2 + r (1/3 - r/4)) (first terms of the series;
 *                                                  dropped terms < 1e-9 relative)
 *      ln x = k ln2 + lg_i + ln(1 + r).
 *    The cell constants are computed in fp64 from a truncated atanh series,
 *    ln v = 2 sum_j s^(2j+1) / (2j+1), s = (v-1)/(v+1) (15 terms, below fp64
 *    rounding for |s| < 0.18), then rounded to fp32.  Every fp32 step is one
 *    IEEE operation (add, multiply or fused multiply-add) in the order
 *    written, so the result is a single well-defined fp32 value.  Valid for
 *    finite normal x > 0, which covers every value the noise definition feeds
 *    it (u in [2^-24, 1-2^-24] and -ln u in [5.9e-8, 16.7]).
 * ------------------------------------------------------------------------- */
static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

#define LOG_CELLS 128
#define LOG_CELLS_BELOW_ONE 76
#define LOG_Z_BASE_BITS 0x3F340000u /* 0.703125 */

static float log_inv[LOG_CELLS];
static float log_lg[LOG_CELLS];
static int log_table_ready = 0;

static double ln_atanh_series(double v)
{
    double s = (v - 1.0) / (v + 1.0);
    double s2 = s * s;
    double acc = 0.0;
    for (int j = 14; j >= 0; --j) acc = acc * s2 + 2.0 / (double)(2 * j + 1);
    return s * acc;
}

static void build_log_table(void)
{
    if (log_table_ready) return;
    for (int i = 0; i < LOG_CELLS; ++i) {
        double lo, width;
        if (i < LOG_CELLS_BELOW_ONE) {
            lo = 0.703125 + (double)i / 256.0;
            width = 1.0 / 256.0;
        } else {
            lo = 1.0 + (double)(i - LOG_CELLS_BELOW_ONE) / 128.0;
            width = 1.0 / 128.0;
        }
        double centre = lo + width / 2.0;
        if (i == LOG_CELLS_BELOW_ONE - 1 || i == LOG_CELLS_BELOW_ONE) {
            log_inv[i] = 1.0f;
            log_lg[i] = 0.0f;
        } else {
            float inv = (float)(1.0 / centre);
            log_inv[i] = inv;
            log_lg[i] = (float)(-ln_atanh_series((double)inv));
        }
    }
    log_table_ready = 1;
}

float oracle_log(float x)
{
    build_log_table();
    const float ln2 = (float)0.69314718055994530941723212145818;
    uint32_t ix = f2u(x);
    uint32_t t = ix - LOG_Z_BASE_BITS;
    int cell = (int)((t >> 16) & (LOG_CELLS - 1));
    int k = (int32_t)t >> 23;                 /* x = z 2^k */
    float z = u2f(ix - (t & 0xFF800000u));
    float r = fmaf(z, log_inv[cell], -1.0f);
    float p = fmaf(r, -0.25f, (float)(1.0 / 3.0));
    p = fmaf(r, p, -0.5f);
    float r2 = r * r;
    float l1p = fmaf(r2, p, r);                /* ln(1 + r) */
    float s = log_lg[cell] + l1p;
    return fmaf((float)k, ln2, s);
}

void oracle_log_array(const float* x, int64_t n, float* out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_log(x[i]);
}

/* Algorithm 1: g = -log(-log u). */
float oracle_gumbel(float u)
{
    float y = -oracle_log(u);
    return -oracle_log(y);
}

void oracle_gumbel_from_words(const uint32_t* words, int64_t n, float* g)
{
    for (int64_t i = 0; i < n; ++i) g[i] = oracle_gumbel(oracle_uniform(words[i]));
}

/* §3.2 / §4.2.2: kappa = phi_bar + g with phi_bar = phi / lambda (§4.2.3). */
static float key_of(float phi, float lambda, uint64_t seed, uint64_t step, uint64_t elem)
{
    float g = oracle_gumbel(oracle_uniform(oracle_philox_word(seed, step, elem)));
    float phi_bar = phi / lambda;
    return phi_bar + g;
}

void oracle_keys(const float* phi, int64_t numel, float lambda, uint64_t seed, uint64_t step,
                 uint64_t elem_offset, float* kappa)
{
    for (int64_t i = 0; i < numel; ++i)
        kappa[i] = key_of(phi[i], lambda, seed, step, elem_offset + (uint64_t)i);
}

/* ------------------------------------------------------------------------- *
 * 3. Hard Gumbel-Top-K (§3.2): pick the largest key, then the largest of the
 *    rest, n times.  A strict '>' keeps the lowest index among equal keys
 *    (fp32 -0 and +0 compare equal).  order[k] is the k-th selected index.
 * ------------------------------------------------------------------------- */
int oracle_topn(const float* kappa, int m, int n, uint8_t* order, uint8_t* hard)
{
    if (m < 1 || m > ORACLE_MAX_M || n < 1 || n > m) return -1;
    int taken[ORACLE_MAX_M];
    for (int j = 0; j < m; ++j) taken[j] = 0;
    for (int k = 0; k < n; ++k) {
        int best = -1;
        for (int j = 0; j < m; ++j) {
            if (taken[j]) continue;
            if (best < 0 || kappa[j] > kappa[best]) best = j;
        }
        taken[best] = 1;
        if (order) order[k] = (uint8_t)best;
    }
    if (hard)
        for (int j = 0; j < m; ++j) hard[j] = (uint8_t)taken[j];
    return 0;
}

/* ------------------------------------------------------------------------- *
 * 4. Relaxation (§3.2 recursion, §4.2.2, Algorithm 1), fp64.
 *    One step: mu = softmax(alpha / tau), evaluated with the largest alpha
 *    subtracted first; omega_i = 1 - mu_i evaluated as sum_{j != i} mu_j;
 *    alpha <- alpha + log(max(omega, FLT_MIN)).  The step record keeps mu,
 *    omega and whether the floor was hit, for the backward.
 * ------------------------------------------------------------------------- */
typedef struct {
    double mu[ORACLE_MAX_M];
    double omega[ORACLE_MAX_M];
    int floored[ORACLE_MAX_M];
} relax_step;

static void softmax_step(const double* alpha, int m, double tau, relax_step* st)
{
    double amax = alpha[0];
    for (int j = 1; j < m; ++j)
        if (alpha[j] > amax) amax = alpha[j];
    double e[ORACLE_MAX_M];
    double total = 0.0;
    for (int j = 0; j < m; ++j) {
        e[j] = exp((alpha[j] - amax) / tau);
        total += e[j];
    }
    for (int i = 0; i < m; ++i) {
        st->mu[i] = e[i] / total;
        double others = 0.0;
        for (int j = 0; j < m; ++j)
            if (j != i) others += e[j];
        st->omega[i] = others / total;
        st->floored[i] = st->omega[i] < (double)FLT_MIN;
    }
}

static void relax_forward(const double* kappa, int m, int n, double tau, relax_step* steps,
                          double* S)
{
    double alpha[ORACLE_MAX_M];
    for (int j = 0; j < m; ++j) {
        alpha[j] = kappa[j]; /* alpha^(1) = kappa */
        if (S) S[j] = 0.0;
    }
    for (int k = 0; k < n; ++k) {
        softmax_step(alpha, m, tau, &steps[k]);
        for (int j = 0; j < m; ++j) {
            if (S) S[j] += steps[k].mu[j];
            double om = steps[k].floored[j] ? (double)FLT_MIN : steps[k].omega[j];
            alpha[j] += log(om);
        }
    }
}

int oracle_relax_fwd(const double* kappa, int m, int n, double tau, double* S)
{
    if (m < 1 || m > ORACLE_MAX_M || n < 1 || n > m || !(tau > 0.0)) return -1;
    relax_step* steps = (relax_step*)malloc(sizeof(relax_step) * (size_t)n);
    if (!steps) return -2;
    relax_forward(kappa, m, n, tau, steps, S);
    free(steps);
    return 0;
}

/* ------------------------------------------------------------------------- *
 * 5. Backward of S = sum_k mu^(k) with respect to kappa (reverse mode).
 *    The paper writes no backward; this is the chain rule through the
 *    recursion of §3.2.  With sbar = dL/dS and a = dL/dalpha^(k+1) carried
 *    down from the later steps (a = 0 above the last step):
 *      mubar_i   = sbar_i - a_i / omega_i         (d log(omega_i)/d mu_i = -1/omega_i;
 *                                                   0 where the floor was hit)
 *      dL/dalpha^(k)_i = a_i + (mu_i / tau) (mubar_i - sum_j mu_j mubar_j)
 *    Because 1 - mu_i = omega_i, the softmax term equals
 *      (mu_i / tau) (omega_i mubar_i - sum_{j != i} mu_j mubar_j),
 *    and omega_i mubar_i = omega_i sbar_i - a_i exactly, so
 *      dL/dalpha^(k)_i = a_i (1 - mu_i / tau) + (mu_i / tau) (omega_i sbar_i - sum_{j != i} mu_j mubar_j)
 *    with 1 - mu_i / tau = (omega_i + (tau - 1)) / tau.  This form never
 *    subtracts two large nearly equal numbers when mu_i is close to 1.
 *    Finally dL/dkappa = dL/dalpha^(1).
 * ------------------------------------------------------------------------- */
static void relax_backward(const relax_step* steps, int m, int n, double tau, const double* sbar,
                           double* dkappa)
{
    double a[ORACLE_MAX_M];
    for (int j = 0; j < m; ++j) a[j] = 0.0;
    for (int k = n - 1; k >= 0; --k) {
        const relax_step* st = &steps[k];
        int has_next = (k < n - 1); /* alpha^(k+1) feeds a later step */
        double mubar[ORACLE_MAX_M];
        for (int j = 0; j < m; ++j) {
            double via_log = (has_next && !st->floored[j]) ? a[j] / st->omega[j] : 0.0;
            mubar[j] = sbar[j] - via_log;
        }
        double a_new[ORACLE_MAX_M];
        for (int i = 0; i < m; ++i) {
            double others = 0.0;
            for (int j = 0; j < m; ++j)
                if (j != i) others += st->mu[j] * mubar[j];
            double soft = (st->mu[i] / tau) * (st->omega[i] * sbar[i] - others);
            double carried = 0.0;
            if (has_next) {
                /* (omega - 1 + tau) / tau, grouped so that tau == 1 gives omega exactly */
                double keep = st->floored[i] ? 1.0 : (st->omega[i] + (tau - 1.0)) / tau;
                carried = a[i] * keep;
            }
            a_new[i] = carried + soft;
        }
        for (int j = 0; j < m; ++j) a[j] = a_new[j];
    }
    for (int j = 0; j < m; ++j) dkappa[j] = a[j];
}

int oracle_relax_bwd(const double* kappa, int m, int n, double tau, const double* sbar,
                     double* dkappa)
{
    if (m < 1 || m > ORACLE_MAX_M || n < 1 || n > m || !(tau > 0.0)) return -1;
    relax_step* steps = (relax_step*)malloc(sizeof(relax_step) * (size_t)n);
    if (!steps) return -2;
    relax_forward(kappa, m, n, tau, steps, NULL);
    relax_backward(steps, m, n, tau, sbar, dkappa);
    free(steps);
    return 0;
}

/* ------------------------------------------------------------------------- *
 * 6. Whole groups.
 * ------------------------------------------------------------------------- */
static float bf16_to_float(uint16_t h)
{
    return u2f((uint32_t)h << 16);
}

static int check_args(int64_t count, int n, int m, float tau, float lambda)
{
    if (count < 0) return -1;
    if (m < 1 || m > ORACLE_MAX_M || n < 1 || n > m) return -1;
    if (!(tau > 0.0f) || !(lambda > 0.0f)) return -1;
    if (!isfinite(tau) || !isfinite(lambda)) return -1;
    return 0;
}

static void group_fwd(const uint16_t* W, const float* phi, int n, int m, float tau,
                      float lambda, uint64_t seed, uint64_t step, uint64_t elem0,
                      uint16_t* Wm, double* S, uint8_t* idx, relax_step* steps)
{
    float kappa[ORACLE_MAX_M] = {0};
    uint8_t order[ORACLE_MAX_M], hard[ORACLE_MAX_M];
    for (int j = 0; j < m; ++j) kappa[j] = key_of(phi[j], lambda, seed, step, elem0 + (uint64_t)j);
    oracle_topn(kappa, m, n, order, hard);
    for (int j = 0; j < m; ++j) Wm[j] = hard[j] ? W[j] : (uint16_t)0x0000u;
    if (idx)
        for (int k = 0; k < n; ++k) idx[k] = order[k];
    if (S) {
        double kd[ORACLE_MAX_M];
        for (int j = 0; j < m; ++j) kd[j] = (double)kappa[j];
        relax_forward(kd, m, n, (double)tau, steps, S);
    }
}

static void group_bwd(const uint16_t* G, const uint16_t* W, const float* phi, int n, int m,
                      float tau, float lambda, uint64_t seed, uint64_t step, uint64_t elem0,
                      double* dphi, relax_step* steps)
{
    double kd[ORACLE_MAX_M] = {0}, sbar[ORACLE_MAX_M] = {0}, dk[ORACLE_MAX_M] = {0};
    for (int j = 0; j < m; ++j) {
        kd[j] = (double)key_of(phi[j], lambda, seed, step, elem0 + (uint64_t)j);
        /* Straight-through: W_masked is used as W (.) S in the backward, so
         * dL/dS = dL/dW_masked (.) W. */
        sbar[j] = (double)bf16_to_float(G[j]) * (double)bf16_to_float(W[j]);
    }
    relax_forward(kd, m, n, (double)tau, steps, NULL);
    relax_backward(steps, m, n, (double)tau, sbar, dk);
    /* kappa = phi / lambda + g, so dL/dphi = dL/dkappa / lambda. */
    for (int j = 0; j < m; ++j) dphi[j] = dk[j] / (double)lambda;
}

int roi_oracle_fwd(const uint16_t* W, const float* logits, int64_t numel, int n, int m,
                   float tau, float lambda, uint64_t seed, uint64_t step, uint64_t elem_offset,
                   uint16_t* W_masked, double* soft_mask, uint8_t* sel_idx)
{
    if (check_args(numel, n, m, tau, lambda) || numel % m != 0) return -1;
    relax_step* steps = (relax_step*)malloc(sizeof(relax_step) * (size_t)n);
    if (!steps) return -2;
    for (int64_t q = 0; q < numel / m; ++q) {
        int64_t base = q * m;
        group_fwd(W + base, logits + base, n, m, tau, lambda, seed, step,
                  elem_offset + (uint64_t)base, W_masked + base,
                  soft_mask ? soft_mask + base : NULL, sel_idx ? sel_idx + q * n : NULL, steps);
    }
    free(steps);
    return 0;
}

int roi_oracle_bwd(const uint16_t* grad_W_masked, const uint16_t* W, const float* logits,
                   int64_t numel, int n, int m, float tau, float lambda, uint64_t seed,
                   uint64_t step, uint64_t elem_offset, double* grad_logits)
{
    if (check_args(numel, n, m, tau, lambda) || numel % m != 0) return -1;
    relax_step* steps = (relax_step*)malloc(sizeof(relax_step) * (size_t)n);
    if (!steps) return -2;
    for (int64_t q = 0; q < numel / m; ++q) {
        int64_t base = q * m;
        group_bwd(grad_W_masked + base, W + base, logits + base, n, m, tau, lambda, seed, step,
                  elem_offset + (uint64_t)base, grad_logits + base, steps);
    }
    free(steps);
    return 0;
}

int roi_oracle_fwd_groups(const uint16_t* W, const float* logits, int64_t ngroups,
                          const uint64_t* group_elem, int n, int m, float tau, float lambda,
                          uint64_t seed, uint64_t step, uint16_t* W_masked, double* soft_mask,
                          uint8_t* sel_idx)
{
    if (check_args(ngroups, n, m, tau, lambda)) return -1;
    relax_step* steps = (relax_step*)malloc(sizeof(relax_step) * (size_t)n);
    if (!steps) return -2;
    for (int64_t q = 0; q < ngroups; ++q) {
        int64_t base = q * m;
        group_fwd(W + base, logits + base, n, m, tau, lambda, seed, step, group_elem[q],
                  W_masked + base, soft_mask ? soft_mask + base : NULL,
                  sel_idx ? sel_idx + q * n : NULL, steps);
    }
    free(steps);
    return 0;
}

int roi_oracle_bwd_groups(const uint16_t* grad_W_masked, const uint16_t* W, const float* logits,
                          int64_t ngroups, const uint64_t* group_elem, int n, int m, float tau,
                          float lambda, uint64_t seed, uint64_t step, double* grad_logits)
{
    if (check_args(ngroups, n, m, tau, lambda)) return -1;
    relax_step* steps = (relax_step*)malloc(sizeof(relax_step) * (size_t)n);
    if (!steps) return -2;
    for (int64_t q = 0; q < ngroups; ++q) {
        int64_t base = q * m;
        group_bwd(grad_W_masked + base, W + base, logits + base, n, m, tau, lambda, seed, step,
                  group_elem[q], grad_logits + base, steps);
    }
    free(steps);
    return 0;
}

/* ------------------------------------------------------------------------- *
 * 7. §4.2.3, exponential annealing:
 *    v_t = max{ v_end, v_init (v_end / v_init)^(t / T_anneal) }.
 * ------------------------------------------------------------------------- */
double oracle_anneal(double v_init, double v_end, double t, double t_anneal)
{
    double v = v_init * pow(v_end / v_init, t / t_anneal);
    return v > v_end ? v : v_end;
}

/* ------------------------------------------------------------------------- *
 * 8. AdamW on the logits (appendix hyperparameters: the logits are trained
 *    with AdamW, beta1 = 0.9, beta2 = 0.95, weight decay 0.05 and a decaying
 *    learning rate; the weights stay frozen).  AdamW is decoupled weight
 *    decay (Loshchilov & Hutter, ICLR 2019) followed by Adam's bias-corrected
 *    moment step (Kingma & Ba, ICLR 2015), at optimizer step t >= 1:
 *        phi <- phi (1 - lr wd)
 *        m   <- beta1 m + (1 - beta1) g
 *        v   <- beta2 v + (1 - beta2) g^2
 *        phi <- phi - lr (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 *    in fp64 from the fp32 state and the fp64 gradient.
 * ------------------------------------------------------------------------- */
int oracle_adamw(const double* grad, int64_t numel, double lr, double beta1, double beta2,
                 double eps, double weight_decay, int64_t t, const float* phi, const float* m,
                 const float* v, double* phi_out, double* m_out, double* v_out)
{
    if (numel < 0 || t < 1 || !(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) ||
        !(eps > 0.0) || !(lr >= 0.0) || !(weight_decay >= 0.0))
        return -1;
    const double bc1 = 1.0 - pow(beta1, (double)t);
    const double bc2 = 1.0 - pow(beta2, (double)t);
    for (int64_t i = 0; i < numel; ++i) {
        const double g = grad[i];
        double p = (double)phi[i] * (1.0 - lr * weight_decay);
        const double mm = beta1 * (double)m[i] + (1.0 - beta1) * g;
        const double vv = beta2 * (double)v[i] + (1.0 - beta2) * g * g;
        p -= lr * (mm / bc1) / (sqrt(vv / bc2) + eps);
        phi_out[i] = p;
        m_out[i] = mm;
        v_out[i] = vv;
    }
    return 0;
}

/* ------------------------------------------------------------------------- *
 * 9. Final mask after training.  The paper anneals the sampling temperature
 *    lambda towards 0 (§4.2.3); as lambda -> 0 the keys phi/lambda + g order
 *    exactly as the logits do, so the sampler's limit is the n largest logits
 *    of each group (ties to the lower index, as in the sampler).  Exported
 *    in the compressed form of a sparse weight: per group the kept weights
 *    and their indices in increasing index order, and for 2:4 the indices as
 *    2-bit fields (group q occupies bits 4(q%8) .. 4(q%8)+3 of word q/8, the
 *    lower kept index in the low two bits).
 * ------------------------------------------------------------------------- */
int oracle_export(const float* logits, const uint16_t* W, int64_t numel, int n, int m,
                  uint16_t* W_masked, uint16_t* values, uint8_t* idx, uint32_t* meta)
{
    if (numel < 0 || m < 1 || m > ORACLE_MAX_M || n < 1 || n > m || numel % m != 0) return -1;
    if (meta && !(n == 2 && m == 4)) return -1;
    const int64_t groups = numel / m;
    if (meta)
        for (int64_t w = 0; w < (groups + 7) / 8; ++w) meta[w] = 0;
    for (int64_t q = 0; q < groups; ++q) {
        uint8_t order[ORACLE_MAX_M], hard[ORACLE_MAX_M];
        oracle_topn(logits + q * m, m, n, order, hard);
        int k = 0;
        for (int j = 0; j < m; ++j) {
            if (W_masked) W_masked[q * m + j] = hard[j] ? W[q * m + j] : (uint16_t)0;
            if (!hard[j]) continue;
            if (values) values[q * n + k] = W[q * m + j];
            if (idx) idx[q * n + k] = (uint8_t)j;
            if (meta) meta[q / 8] |= (uint32_t)j << (4 * (q % 8) + 2 * k);
            ++k;
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------- *
 * 10. The categorical mask sampler the paper compares with (appendix,
 *     "Optimization Efficiency": one logit alpha_c per feasible n-hot mask c
 *     of a group, Pr(c) = softmax(alpha)_c, sampled by Gumbel-Softmax).
 *     Readings (shared with the kernels):
 *     - the C = binom(m, n) candidates are the n-subsets of {0..m-1} in
 *       lexicographic order;
 *     - keys kappa_c = fl(fl(alpha_c / lambda) + g_c), as for the item
 *       logits; candidate c of global group Q draws the noise of element
 *       index 4 B Q + c, B = ceil(C / 4) (each group starts a Philox block);
 *     - the hard sample is the candidate of largest key (ties to the lower
 *       candidate index); W_masked = W (.) that mask;
 *     - relaxed: y = softmax(kappa / tau) and S_j = sum_c y_c [j in c];
 *     - backward (straight-through, as for the item logits): sbar = G (.) W,
 *       ybar_c = sum_{j in c} sbar_j, dL/dkappa = y (.) (ybar - <y, ybar>) / tau,
 *       dL/dalpha = dL/dkappa / lambda.
 * ------------------------------------------------------------------------- */
#define ORACLE_MAX_CAT 70

int oracle_cat_candidates(int n, int m, uint32_t* masks)
{
    if (m < 1 || m > 8 || n < 1 || n > m) return -1;
    int count = 0;
    for (uint32_t bits = 0; bits < (1u << m); ++bits) {
        int pop = 0;
        for (int j = 0; j < m; ++j) pop += (bits >> j) & 1u;
        if (pop == n) ++count;
    }
    /* lexicographic order of the index sets: walk the combinations directly */
    int idx[8], c = 0;
    for (int k = 0; k < n; ++k) idx[k] = k;
    for (;;) {
        uint32_t mask = 0;
        for (int k = 0; k < n; ++k) mask |= 1u << idx[k];
        if (masks) masks[c] = mask;
        ++c;
        int k = n - 1;
        while (k >= 0 && idx[k] == m - n + k) --k;
        if (k < 0) break;
        ++idx[k];
        for (int r = k + 1; r < n; ++r) idx[r] = idx[r - 1] + 1;
    }
    return c == count ? c : -1;
}

static int cat_group_keys(const float* alpha, int C, float lambda, uint64_t seed, uint64_t step,
                          uint64_t Q, float* kappa)
{
    const uint64_t B = (uint64_t)(C + 3) / 4;
    int best = 0;
    for (int c = 0; c < C; ++c) {
        kappa[c] = key_of(alpha[c], lambda, seed, step, 4 * B * Q + (uint64_t)c);
        if (kappa[c] > kappa[best]) best = c; /* strict: ties keep the lower index */
    }
    return best;
}

static void cat_softmax(const float* kappa, int C, double tau, double* y)
{
    double mx = kappa[0];
    for (int c = 1; c < C; ++c) mx = kappa[c] > mx ? kappa[c] : mx;
    double t = 0.0;
    for (int c = 0; c < C; ++c) {
        y[c] = exp(((double)kappa[c] - mx) / tau);
        t += y[c];
    }
    for (int c = 0; c < C; ++c) y[c] /= t;
}

int oracle_cat_fwd(const uint16_t* W, const float* alpha, int64_t ngroups, int n, int m,
                   float tau, float lambda, uint64_t seed, uint64_t step, uint64_t group_offset,
                   uint16_t* W_masked, double* S, uint8_t* choice)
{
    uint32_t masks[ORACLE_MAX_CAT];
    if (check_args(ngroups, n, m, tau, lambda)) return -1;
    const int C = oracle_cat_candidates(n, m, masks);
    if (C < 1 || C > ORACLE_MAX_CAT) return -1;
    for (int64_t q = 0; q < ngroups; ++q) {
        float kappa[ORACLE_MAX_CAT];
        const int best = cat_group_keys(alpha + q * C, C, lambda, seed, step,
                                        group_offset + (uint64_t)q, kappa);
        if (choice) choice[q] = (uint8_t)best;
        for (int j = 0; j < m; ++j)
            if (W_masked)
                W_masked[q * m + j] = ((masks[best] >> j) & 1u) ? W[q * m + j] : (uint16_t)0;
        if (S) {
            double y[ORACLE_MAX_CAT];
            cat_softmax(kappa, C, (double)tau, y);
            for (int j = 0; j < m; ++j) {
                double acc = 0.0;
                for (int c = 0; c < C; ++c)
                    if ((masks[c] >> j) & 1u) acc += y[c];
                S[q * m + j] = acc;
            }
        }
    }
    return 0;
}

int oracle_cat_bwd(const uint16_t* G, const uint16_t* W, const float* alpha, int64_t ngroups,
                   int n, int m, float tau, float lambda, uint64_t seed, uint64_t step,
                   uint64_t group_offset, double* dalpha)
{
    uint32_t masks[ORACLE_MAX_CAT];
    if (check_args(ngroups, n, m, tau, lambda)) return -1;
    const int C = oracle_cat_candidates(n, m, masks);
    if (C < 1 || C > ORACLE_MAX_CAT) return -1;
    for (int64_t q = 0; q < ngroups; ++q) {
        float kappa[ORACLE_MAX_CAT];
        double y[ORACLE_MAX_CAT], ybar[ORACLE_MAX_CAT], sbar[8];
        cat_group_keys(alpha + q * C, C, lambda, seed, step, group_offset + (uint64_t)q, kappa);
        cat_softmax(kappa, C, (double)tau, y);
        for (int j = 0; j < m; ++j)
            sbar[j] = (double)bf16_to_float(G[q * m + j]) * (double)bf16_to_float(W[q * m + j]);
        double dot = 0.0;
        for (int c = 0; c < C; ++c) {
            ybar[c] = 0.0;
            for (int j = 0; j < m; ++j)
                if ((masks[c] >> j) & 1u) ybar[c] += sbar[j];
            dot += y[c] * ybar[c];
        }
        for (int c = 0; c < C; ++c)
            dalpha[q * C + c] = y[c] * (ybar[c] - dot) / (double)tau / (double)lambda;
    }
    return 0;
}

/* ------------------------------------------------------------------------- *
 * 11. The whole-array forward and backward on several threads.  Groups are
 *     independent (§4.1: each group of m weights gets its own mask; the noise
 *     of an element depends only on its global index), so the groups are cut
 *     into contiguous ranges, one per POSIX thread, and each thread runs the
 *     scalar per-group code above on its range.  The outputs are the same
 *     bits for every thread count.  Also the relaxation's backward on given
 *     keys over many groups (the tests' fp32 rounding allowance).
 * ------------------------------------------------------------------------- */
typedef struct {
    int kind; /* 0 forward, 1 backward, 2 relaxation backward on given keys */
    int64_t g0, g1;
    const uint16_t *W, *G;
    const float* logits;
    const double *kappa, *sbar;
    int n, m;
    float tau, lambda;
    double tau64; /* the relaxation's temperature for kind 2 */
    uint64_t seed, step, elem_offset;
    uint16_t* Wm;
    double *S, *out;
    uint8_t* idx;
    int status;
} mt_job;

static void* mt_run(void* arg)
{
    mt_job* j = (mt_job*)arg;
    relax_step* steps = (relax_step*)malloc(sizeof(relax_step) * (size_t)j->n);
    if (!steps) {
        j->status = -2;
        return NULL;
    }
    const int m = j->m;
    for (int64_t q = j->g0; q < j->g1; ++q) {
        const int64_t base = q * m;
        if (j->kind == 0) {
            group_fwd(j->W + base, j->logits + base, j->n, m, j->tau, j->lambda, j->seed, j->step,
                      j->elem_offset + (uint64_t)base, j->Wm + base, j->S ? j->S + base : NULL,
                      j->idx ? j->idx + q * j->n : NULL, steps);
        } else if (j->kind == 1) {
            group_bwd(j->G + base, j->W + base, j->logits + base, j->n, m, j->tau, j->lambda,
                      j->seed, j->step, j->elem_offset + (uint64_t)base, j->out + base, steps);
        } else {
            relax_forward(j->kappa + base, m, j->n, j->tau64, steps, NULL);
            relax_backward(steps, m, j->n, j->tau64, j->sbar + base, j->out + base);
        }
    }
    free(steps);
    j->status = 0;
    return NULL;
}

static int mt_launch(mt_job proto, int64_t ngroups, int threads)
{
    if (threads < 1) threads = 1;
    if (threads > 256) threads = 256;
    if ((int64_t)threads > ngroups) threads = ngroups > 0 ? (int)ngroups : 1;
    mt_job jobs[256];
    pthread_t tid[256];
    int started[256];
    int status = 0;
    for (int t = 0; t < threads; ++t) {
        jobs[t] = proto;
        jobs[t].g0 = ngroups * t / threads;
        jobs[t].g1 = ngroups * (t + 1) / threads;
        jobs[t].status = -3;
        started[t] = pthread_create(&tid[t], NULL, mt_run, &jobs[t]) == 0;
        if (!started[t]) mt_run(&jobs[t]); /* run it here instead */
    }
    for (int t = 0; t < threads; ++t) {
        if (started[t]) pthread_join(tid[t], NULL);
        if (jobs[t].status) status = jobs[t].status;
    }
    return status;
}

int roi_oracle_fwd_mt(const uint16_t* W, const float* logits, int64_t numel, int n, int m,
                      float tau, float lambda, uint64_t seed, uint64_t step, uint64_t elem_offset,
                      uint16_t* W_masked, double* soft_mask, uint8_t* sel_idx, int threads)
{
    if (check_args(numel, n, m, tau, lambda) || numel % m != 0) return -1;
    mt_job j;
    memset(&j, 0, sizeof j);
    j.kind = 0;
    j.W = W;
    j.logits = logits;
    j.n = n;
    j.m = m;
    j.tau = tau;
    j.lambda = lambda;
    j.seed = seed;
    j.step = step;
    j.elem_offset = elem_offset;
    j.Wm = W_masked;
    j.S = soft_mask;
    j.idx = sel_idx;
    return mt_launch(j, numel / m, threads);
}

int roi_oracle_bwd_mt(const uint16_t* grad_W_masked, const uint16_t* W, const float* logits,
                      int64_t numel, int n, int m, float tau, float lambda, uint64_t seed,
                      uint64_t step, uint64_t elem_offset, double* grad_logits, int threads)
{
    if (check_args(numel, n, m, tau, lambda) || numel % m != 0) return -1;
    mt_job j;
    memset(&j, 0, sizeof j);
    j.kind = 1;
    j.G = grad_W_masked;
    j.W = W;
    j.logits = logits;
    j.n = n;
    j.m = m;
    j.tau = tau;
    j.lambda = lambda;
    j.seed = seed;
    j.step = step;
    j.elem_offset = elem_offset;
    j.out = grad_logits;
    return mt_launch(j, numel / m, threads);
}

int oracle_relax_bwd_groups(const double* kappa, int64_t ngroups, int m, int n, double tau,
                            const double* sbar, double* dkappa, int threads)
{
    if (ngroups < 0 || m < 1 || m > ORACLE_MAX_M || n < 1 || n > m || !(tau > 0.0)) return -1;
    mt_job j;
    memset(&j, 0, sizeof j);
    j.kind = 2;
    j.kappa = kappa;
    j.sbar = sbar;
    j.n = n;
    j.m = m;
    j.tau64 = tau;
    j.out = dkappa;
    return mt_launch(j, ngroups, threads);
}
