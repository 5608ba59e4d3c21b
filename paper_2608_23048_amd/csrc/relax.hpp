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

// Relaxation (§3.2 recursion, Algorithm 1) in fp32:
//   alpha^(1) = kappa; mu^(k) = softmax(alpha^(k) / tau);
//   alpha^(k+1) = alpha^(k) + log(1 - mu^(k));  S = sum_k mu^(k).
// Internally b = (alpha - max kappa) * log2(e) / tau, so the softmax is
// exp2(b - max b) and the update is b += log2(1 - mu) / tau: the same values
// with one multiply fewer per element and step.  Subtracting the group's
// largest key first keeps the competing entries near 0, where fp32 is
// densest.  1 - mu_j is evaluated as (sum of the other exponentials) / total,
// which never cancels, and log(1 - mu) is floored at log(FLT_MIN).
// key_scale turns key differences into b: log2(e) / tau for keys in natural
// units, 1 / tau for keys already in log2 units (any common offset cancels).
template <int M, int N, bool kWantS, bool kKeep>
__device__ __forceinline__ void relax_forward(const float (&kappa)[M], float key_scale,
                                              float inv_tau, float (&S)[M], StepRec<M> (&rec)[N])
{
    float kmax = kappa[0];
#pragma unroll
    for (int j = 1; j < M; ++j) kmax = fmaxf(kmax, kappa[j]);
    const float c = key_scale;
    float b[M];
#pragma unroll
    for (int j = 0; j < M; ++j) {
        b[j] = (kappa[j] - kmax) * c;
        if (kWantS) S[j] = 0.0f;
    }
#pragma unroll
    for (int k = 0; k < N; ++k) {
        float e[M];
        if (k == 0) { // the largest b is exactly 0
#pragma unroll
            for (int j = 0; j < M; ++j) e[j] = __builtin_amdgcn_exp2f(b[j]);
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
            if (kWantS) S[j] += mu;
            if (kKeep) {
                rec[k].mu[j] = mu;
                rec[k].om[j] = om;
            }
            if (k + 1 < N)
                b[j] = __builtin_fmaf(__builtin_amdgcn_logf(fmaxf(om, kFltMin)), inv_tau, b[j]);
        }
    }
}

// Reverse sweep of relax_forward: given sbar = dL/dS, returns dL/dkappa.
// Chain rule through the recursion, with a = dL/dalpha^(k+1) (0 above the
// last step) and omega = 1 - mu^(k):
//   mubar_j = sbar_j - a_j / omega_j            (no a_j / omega_j where the floor was hit)
//   dL/dalpha^(k)_j = a_j + (mu_j / tau) (mubar_j - sum_l mu_l mubar_l).
// With 1 - mu_j = omega_j and omega_j mubar_j = omega_j sbar_j - a_j this is
//   dL/dalpha^(k)_j = a_j keep_j + (mu_j / tau) (omega_j sbar_j - sum_{l != j} mu_l mubar_l),
//   keep_j = 1 - mu_j / tau = (omega_j + tau - 1) / tau   (1 where the floor was hit),
// the same form for every j, with no difference of two large numbers when
// mu_j is close to 1 (the sum over l != j is built from prefix and suffix
// sums).
template <int M, int N>
__device__ __forceinline__ void relax_backward(const StepRec<M> (&rec)[N], const float (&sbar)[M],
                                               float tau, float inv_tau, float (&abar)[M])
{
    const float keep0 = (tau - 1.0f) * inv_tau;
#pragma unroll
    for (int k = N - 1; k >= 0; --k) {
        const bool has_next = (k + 1 < N);
        float t[M];
#pragma unroll
        for (int j = 0; j < M; ++j) {
            float mubar = sbar[j];
            if (has_next) {
                const float om = rec[k].om[j];
                const float r = abar[j] * __builtin_amdgcn_rcpf(om);
                mubar = (om >= kFltMin) ? mubar - r : mubar;
            }
            t[j] = rec[k].mu[j] * mubar;
        }
        float q[M], unused;
        sums_but_one<M>(t, q, unused);
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const float om = rec[k].om[j];
            const float inner = __builtin_fmaf(om, sbar[j], -q[j]);
            const float m_t = rec[k].mu[j] * inv_tau;
            float carry = 0.0f;
            if (has_next) {
                // keep = 1 - mu/tau, from mu while mu < 1/2 and from omega above (where
                // 1 - mu would cancel); 1 where the floor was hit
                const float mu = rec[k].mu[j];
                float keep = mu < 0.5f ? __builtin_fmaf(-mu, inv_tau, 1.0f)
                                       : __builtin_fmaf(om, inv_tau, keep0);
                keep = (om >= kFltMin) ? keep : 1.0f;
                carry = abar[j] * keep;
            }
            abar[j] = __builtin_fmaf(m_t, inner, carry);
        }
    }
}

} // namespace roi
