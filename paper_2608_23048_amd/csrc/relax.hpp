// relax.hpp -- per-group hard top-n, Gumbel-Top-K relaxation and its reverse
// sweep, on register arrays of one group (m keys held by one lane).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace roi {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kFltMin = 1.17549435e-38f;

// Hard Gumbel-Top-K (§3.2): rank_j = number of keys that beat key j, where
// i beats j when kappa_i > kappa_j, or kappa_i == kappa_j and i < j.  The n
// keys of rank < n are kept; rank is also the selection order.
template <int M>
__device__ __forceinline__ void rank_keys(const float (&kappa)[M], int (&rank)[M])
{
#pragma unroll
    for (int j = 0; j < M; ++j) rank[j] = 0;
#pragma unroll
    for (int i = 0; i < M; ++i) {
#pragma unroll
        for (int j = i + 1; j < M; ++j) {
            const bool i_wins = kappa[i] >= kappa[j];
            rank[j] += i_wins ? 1 : 0;
            rank[i] += i_wins ? 0 : 1;
        }
    }
}

// Hard top-n of four keys through a 64-entry table.  The six pairwise
// comparisons c_ij = (kappa_i >= kappa_j), i < j (ties to the lower index),
// form a 6-bit code; since >= on finite floats is transitive, the code fixes
// every rank (rank_j = number of entries that beat j).  Entry `code` holds the
// two bf16-pair masks that keep the entries of rank < n, and the selection
// order packed one index per byte.
struct Top4Entry {
    uint32_t m01, m23, order, unused;
};

struct Top4Table {
    Top4Entry e[64];
};

constexpr Top4Table make_top4_table(int n)
{
    Top4Table t{};
    for (int code = 0; code < 64; ++code) {
        const int c01 = code & 1, c02 = (code >> 1) & 1, c03 = (code >> 2) & 1;
        const int c12 = (code >> 3) & 1, c13 = (code >> 4) & 1, c23 = (code >> 5) & 1;
        const int rank[4] = {(1 - c01) + (1 - c02) + (1 - c03), c01 + (1 - c12) + (1 - c13),
                             c02 + c12 + (1 - c23), c03 + c13 + c23};
        uint32_t m01 = 0, m23 = 0, order = 0;
        if (rank[0] < n) m01 |= 0x0000FFFFu;
        if (rank[1] < n) m01 |= 0xFFFF0000u;
        if (rank[2] < n) m23 |= 0x0000FFFFu;
        if (rank[3] < n) m23 |= 0xFFFF0000u;
        for (int j = 0; j < 4; ++j)
            if (rank[j] < n) order |= (uint32_t)j << (8 * rank[j]);
        t.e[code].m01 = m01;
        t.e[code].m23 = m23;
        t.e[code].order = order;
        t.e[code].unused = 0;
    }
    return t;
}

template <int N>
__device__ const Top4Table kTop4Table = make_top4_table(N);

__device__ __forceinline__ uint32_t top4_code(const float (&k)[4])
{
    return (k[0] >= k[1] ? 1u : 0u) | (k[0] >= k[2] ? 2u : 0u) | (k[0] >= k[3] ? 4u : 0u) |
           (k[1] >= k[2] ? 8u : 0u) | (k[1] >= k[3] ? 16u : 0u) | (k[2] >= k[3] ? 32u : 0u);
}

// Sums over "all entries but j" for every j, from prefix and suffix sums
// (no subtraction, so a dominant entry never cancels the others away).
template <int M>
__device__ __forceinline__ void sums_but_one(const float (&x)[M], float (&out)[M], float& total)
{
    if constexpr (M == 4) { // pair sums: six adds, seven with the total
        const float pa = x[0] + x[1], pb = x[2] + x[3];
        out[0] = x[1] + pb;
        out[1] = x[0] + pb;
        out[2] = pa + x[3];
        out[3] = pa + x[2];
        total = pa + pb;
        return;
    }
    float pre[M], suf[M];
    pre[0] = x[0];
#pragma unroll
    for (int j = 1; j < M; ++j) pre[j] = pre[j - 1] + x[j];
    suf[M - 1] = x[M - 1];
#pragma unroll
    for (int j = M - 2; j >= 0; --j) suf[j] = suf[j + 1] + x[j];
    out[0] = suf[1];
    out[M - 1] = pre[M - 2];
#pragma unroll
    for (int j = 1; j < M - 1; ++j) out[j] = pre[j - 1] + suf[j + 1];
    total = pre[M - 1];
}

// One record per relaxation step, kept for the reverse sweep.
template <int M>
struct StepRec {
    float mu[M]; // mu^(k)
    float om[M]; // 1 - mu^(k), evaluated as the sum of the other entries over the total
};

// Keys scaled for the relaxation: b_j = kappa_j * key_scale, the softmax
// argument alpha / tau in log2 units; bmax = max b.  Returns the span
// (max - min) of b.  key_scale is log2(e) / tau for keys in natural units and
// 1 / tau for keys already in log2 units (any common offset cancels).  The
// keys are not shifted by their maximum here: each softmax subtracts the
// largest b of its own step, so the entries that compete at a step are
// compared without the rounding of a shift by an entry already selected
// (which would cost about ulp(span) in every exponent).
template <int M, bool kSpan = true>
__device__ __forceinline__ float scaled_keys(const float (&kappa)[M], float key_scale, float (&b)[M],
                                             float& bmax)
{
    float kmax = kappa[0], kmin = kappa[0];
#pragma unroll
    for (int j = 1; j < M; ++j) {
        kmax = fmaxf(kmax, kappa[j]);
        if (kSpan) kmin = fminf(kmin, kappa[j]);
    }
#pragma unroll
    for (int j = 0; j < M; ++j) b[j] = kappa[j] * key_scale;
    bmax = kmax * key_scale; // = max b (rounding is monotone)
    return kSpan ? (kmax - kmin) * key_scale : 0.0f;
}

// Relaxation (§3.2 recursion, Algorithm 1) in fp32:
//   alpha^(1) = kappa; mu^(k) = softmax(alpha^(k) / tau);
//   alpha^(k+1) = alpha^(k) + log(1 - mu^(k));  S = sum_k mu^(k).
// Internally b = alpha * log2(e) / tau (scaled_keys), so the softmax is
// exp2(b - max b) and the update is b += log2(1 - mu) / tau: the same values
// with one multiply fewer per element and step.  1 - mu_j is evaluated as
// (sum of the other exponentials) / total, which never cancels, and
// log(1 - mu) is floored at log(FLT_MIN).  The records of the updating steps
// hold max(1 - mu, FLT_MIN), the value whose log was taken: a floored entry
// shows as exactly FLT_MIN (relax_backward).
template <int M, int N, bool kWantS, bool kKeep>
__device__ __forceinline__ void relax_forward(float (&b)[M], float bmax0, float inv_tau,
                                              float (&S)[M], StepRec<M> (&rec)[N])
{
#pragma unroll
    for (int j = 0; j < M; ++j)
        if (kWantS) S[j] = 0.0f;
#pragma unroll
    for (int k = 0; k < N; ++k) {
        float e[M];
        if (k == 0) { // the largest b is known
#pragma unroll
            for (int j = 0; j < M; ++j) e[j] = __builtin_amdgcn_exp2f(b[j] - bmax0);
        } else {
            float bmax = b[0];
#pragma unroll
            for (int j = 1; j < M; ++j) bmax = fmaxf(bmax, b[j]);
#pragma unroll
            for (int j = 0; j < M; ++j) e[j] = __builtin_amdgcn_exp2f(b[j] - bmax);
        }
        float others[M], total;
        sums_but_one<M>(e, others, total);
        const float inv_total = __builtin_amdgcn_rcpf(total);
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const float mu = e[j] * inv_total;
            const float om = others[j] * inv_total;
            const float om_floor = k + 1 < N ? fmaxf(om, kFltMin) : om;
            if (kWantS) S[j] += mu;
            if (kKeep) {
                rec[k].mu[j] = mu;
                rec[k].om[j] = om_floor;
            }
            if (k + 1 < N) b[j] = __builtin_fmaf(__builtin_amdgcn_logf(om_floor), inv_tau, b[j]);
        }
    }
}

// The same recursion on the exponentials.  With e proportional to
// exp(alpha / tau), the update alpha += log(1 - mu) is e <- e * (1 - mu)^q,
// q = 1 / tau; rescaled by the total this is e <- mu * omega^q: no maximum,
// shift or floor per element and step, and for tau = 1 (kQ = 1) or 1/2
// (kQ = 2) no log or exp either (a product of q + 1 factors).  Other
// temperatures (kQ = 0) take omega^q = exp2(q log2 omega).
//
// When it agrees with relax_forward: call an entry "dominant" at a step where
// its mu >= 1/2 (at most one entry per step).  An entry never dominant so far
// has omega > 1/2, so each step multiplies its weight by at least 2^-q while
// the total of the products never exceeds 1: after k steps its mu is at least
// 2^-(span + log2 M + k q).  Before the last step at most N - 1 <= M - 1
// entries have been dominant, so one such entry always exists, and the
// dominant entry's omega (the sum of the others) is at least as large.  Hence
// span + log2 M + (N - 1) q <= kExpNormalBound keeps every such mu and omega
// above 2^-91: normal numbers far from underflow, and far above the FLT_MIN
// floor of log(1 - mu), which is therefore never reached.  An entry that has
// been dominant and falls below 2^-126 moves the total by less than 2^-35 of
// itself, so the exp-domain and log-domain recursions agree to rounding.
// Unlike the log-domain loop, this form keeps the first step's shift by the
// largest key for good: each exponent b_j - bmax carries a rounding of about
// 2^-24 |b_j - bmax| (with that of key_scale), a relative error of about
// 4e-8 span in e_j.  span <= kExpSpanAccuracy keeps it near 1e-6.
constexpr float kExpNormalBound = 91.0f;
constexpr float kExpSpanAccuracy = 32.0f;

template <int kQ>
__device__ __forceinline__ float pow_q(float om, float q)
{
    if constexpr (kQ == 1) return om;
    else if constexpr (kQ == 2) return om * om;
    else return __builtin_amdgcn_exp2f(__builtin_amdgcn_logf(om) * q);
}

template <int M, int N, bool kWantS, bool kKeep, int kQ>
__device__ __forceinline__ void relax_forward_exp(const float (&b)[M], float bmax, float q,
                                                  float (&S)[M], StepRec<M> (&rec)[N])
{
    static_assert(kQ >= 0 && kQ <= 2, "exp-domain recursion: kQ");
    float e[M];
#pragma unroll
    for (int j = 0; j < M; ++j) {
        e[j] = __builtin_amdgcn_exp2f(b[j] - bmax);
        if (kWantS) S[j] = 0.0f;
    }
#pragma unroll
    for (int k = 0; k < N; ++k) {
        float others[M], total;
        sums_but_one<M>(e, others, total);
        const float inv_total = __builtin_amdgcn_rcpf(total);
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const float mu = e[j] * inv_total;
            const float om = others[j] * inv_total;
            if (kWantS) S[j] += mu;
            if (kKeep) {
                rec[k].mu[j] = mu;
                rec[k].om[j] = om;
            }
            if (k + 1 < N) e[j] = mu * pow_q<kQ>(om, q);
        }
    }
}

// Reverse sweep of relax_forward / relax_forward_exp: given sbar = dL/dS,
// returns dL/dkappa for kappa in natural units (the records are unit-free, so
// the units the caller's keys had when forming b do not matter; the 1/tau is
// that of softmax(alpha / tau)).  Chain rule through the recursion, with a = dL/dalpha^(k+1)
// (0 above the last step), omega = 1 - mu^(k),
//   mubar_j = sbar_j - a_j / omega_j,
//   dL/dalpha^(k)_j = a_j + (mu_j / tau) (mubar_j - sum_l mu_l mubar_l).
// Since omega_j mubar_j = omega_j sbar_j - a_j, with
// X_j = omega_j sbar_j - sum_{l != j} mu_l mubar_l this is
//   dL/dalpha^(k)_j = a_j + (mu_j / tau) (X_j - a_j),
// one form for every j, and the sum over l != j comes from prefix and suffix
// sums (nothing cancels when mu_j is near 1).  The rounding of X_j - a_j is
// relative to |a_j|, which is small exactly for an entry whose mu is near 1:
// that entry is selected at this step, so its later weights, and with them
// a_j, are negligible.
// With kFloor, an entry whose 1 - mu fell below FLT_MIN at an updating step
// had its log floored, so no derivative flows through it: mubar_j = sbar_j and
// dL/dalpha^(k)_j = a_j + (mu_j / tau) X_j.  The records of relax_forward hold
// max(1 - mu, FLT_MIN) there, so such an entry reads exactly FLT_MIN: it takes
// a_j = 0 in both places, which also keeps a_j / omega_j finite.  X_j then uses
// FLT_MIN for an omega_j below it, a change below FLT_MIN |sbar_j|.  Without
// kFloor the caller has ruled the floor out (the exp-domain form's span
// bound, whose records hold 1 - mu itself).
template <int M, int N, bool kTauIsOne, bool kFloor>
__device__ __forceinline__ void relax_backward(const StepRec<M> (&rec)[N], const float (&sbar)[M],
                                               float inv_tau, float (&abar)[M])
{
#pragma unroll
    for (int k = N - 1; k >= 0; --k) {
        const bool has_next = (k + 1 < N);
        float t[M], a_in[M];
#pragma unroll
        for (int j = 0; j < M; ++j) {
            float mubar = sbar[j];
            a_in[j] = 0.0f;
            if (has_next) {
                const float om = rec[k].om[j];
                a_in[j] = !kFloor || om > kFltMin ? abar[j] : 0.0f;
                mubar = __builtin_fmaf(-a_in[j], __builtin_amdgcn_rcpf(om), sbar[j]);
            }
            t[j] = rec[k].mu[j] * mubar;
        }
        float q[M], unused;
        sums_but_one<M>(t, q, unused);
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const float x = __builtin_fmaf(rec[k].om[j], sbar[j], -q[j]);
            const float m_t = kTauIsOne ? rec[k].mu[j] : rec[k].mu[j] * inv_tau;
            abar[j] = has_next ? __builtin_fmaf(m_t, x - a_in[j], abar[j]) : m_t * x;
        }
    }
}

} // namespace roi
