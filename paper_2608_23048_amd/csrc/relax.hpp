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

// One record per relaxation step, kept for the reverse sweep.
template <int M>
struct StepRec {
    float mu[M];   // mu^(k)
    float om_star; // 1 - mu^(k)_{i*}, evaluated as the sum of the other entries
    int istar;     // index of the largest adjusted key at step k
};

// Relaxation (§3.2 recursion, Algorithm 1) in fp32:
//   alpha^(1) = kappa; mu^(k) = softmax(alpha^(k) / tau);
//   alpha^(k+1) = alpha^(k) + log(1 - mu^(k));  S = sum_k mu^(k).
// Internally b = (alpha - max kappa) * log2(e) / tau, so the softmax is
// exp2(b - max b) and the update is b += log2(1 - mu) / tau: the same values
// with one multiply fewer per element and step.  Subtracting the group's
// largest key first keeps the competing entries near 0, where fp32 is
// densest, and makes b = 0 exactly at the first argmax.
// 1 - mu_i: for i != i* it is >= 1/2, so 1 - mu_i loses nothing; for the
// current argmax i* it is rest / T with rest = the sum of the other
// exponentials (no cancellation).  log(1 - mu) is floored at log(FLT_MIN).
template <int M, int N, bool kWantS, bool kKeep>
__device__ __forceinline__ void relax_forward(const float (&kappa)[M], float inv_tau,
                                              float (&S)[M], StepRec<M> (&rec)[N])
{
    float kmax = kappa[0];
    int istar = 0;
#pragma unroll
    for (int j = 1; j < M; ++j) {
        const bool gt = kappa[j] > kmax;
        kmax = gt ? kappa[j] : kmax;
        istar = gt ? j : istar;
    }
    const float c = kLog2e * inv_tau;
    float b[M];
#pragma unroll
    for (int j = 0; j < M; ++j) {
        b[j] = (kappa[j] - kmax) * c;
        if (kWantS) S[j] = 0.0f;
    }
#pragma unroll
    for (int k = 0; k < N; ++k) {
        float bmax = 0.0f; // step 1: b[istar] == 0 exactly
        if (k > 0) {
            bmax = b[0];
            istar = 0;
#pragma unroll
            for (int j = 1; j < M; ++j) {
                const bool gt = b[j] > bmax;
                bmax = gt ? b[j] : bmax;
                istar = gt ? j : istar;
            }
        }
        float e[M];
        float rest = 0.0f;
#pragma unroll
        for (int j = 0; j < M; ++j) {
            e[j] = __builtin_amdgcn_exp2f(k > 0 ? b[j] - bmax : b[j]); // e[istar] == 1 exactly
            rest += (j == istar) ? 0.0f : e[j];
        }
        const float inv_total = __builtin_amdgcn_rcpf(1.0f + rest);
        const float om_star = rest * inv_total;
        float mu[M];
#pragma unroll
        for (int j = 0; j < M; ++j) {
            mu[j] = e[j] * inv_total;
            if (kWantS) S[j] += mu[j];
            if (kKeep) rec[k].mu[j] = mu[j];
        }
        if (kKeep) {
            rec[k].om_star = om_star;
            rec[k].istar = istar;
        }
        if (k + 1 < N) {
            const float om_star_f = fmaxf(om_star, kFltMin);
#pragma unroll
            for (int j = 0; j < M; ++j) {
                const float om = (j == istar) ? om_star_f : 1.0f - mu[j];
                b[j] = __builtin_fmaf(__builtin_amdgcn_logf(om), inv_tau, b[j]);
            }
        }
    }
}

// Reverse sweep of relax_forward: given sbar = dL/dS, returns dL/dkappa.
// Chain rule through the recursion, with a = dL/dalpha^(k+1) (0 above the
// last step), omega = 1 - mu^(k):
//   mubar_i = sbar_i - a_i / omega_i          (0 instead where the floor was hit)
//   dL/dalpha^(k)_i = a_i + (mu_i / tau) (mubar_i - sum_j mu_j mubar_j).
// For i != i* this is evaluated as written (mu_i <= 1/2, omega_i >= 1/2).  For
// i* the product mu_i* * (...) may cancel catastrophically when mu_i* ~ 1, so
// the identity omega_i* mubar_i* = omega_i* sbar_i* - a_i* is used:
//   dL/dalpha^(k)_i* = a_i* (omega* + tau - 1) / tau
//                      + (mu_i* / tau) (omega* sbar_i* - sum_{j != i*} mu_j mubar_j).
// A floored omega* is replaced by +inf, so that a_i* / omega* = 0.
template <int M, int N>
__device__ __forceinline__ void relax_backward(const StepRec<M> (&rec)[N], const float (&sbar)[M],
                                               float tau, float inv_tau, float (&abar)[M])
{
#pragma unroll
    for (int j = 0; j < M; ++j) abar[j] = 0.0f;
#pragma unroll
    for (int k = N - 1; k >= 0; --k) {
        const bool has_next = (k + 1 < N);
        const int istar = rec[k].istar;
        const float oms = rec[k].om_star;
        const bool floored = !(oms >= kFltMin);
        float t[M];
        float p_all = 0.0f, p_excl = 0.0f, sbar_is = 0.0f, abar_is = 0.0f;
        float mubar[M];
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const bool is = (j == istar);
            const float mu = rec[k].mu[j];
            mubar[j] = sbar[j];
            if (has_next) {
                const float om = is ? (floored ? __builtin_inff() : oms) : 1.0f - mu;
                mubar[j] = __builtin_fmaf(-abar[j], __builtin_amdgcn_rcpf(om), sbar[j]);
            }
            t[j] = mu * mubar[j];
            p_all += t[j];
            p_excl += is ? 0.0f : t[j];
            sbar_is = is ? sbar[j] : sbar_is;
            if (has_next) abar_is = is ? abar[j] : abar_is;
        }
        const float inner_is = __builtin_fmaf(oms, sbar_is, -p_excl);
        float carry_is = 0.0f;
        if (has_next) carry_is = abar_is * (floored ? 1.0f : (oms + (tau - 1.0f)) * inv_tau);
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const bool is = (j == istar);
            const float m_t = rec[k].mu[j] * inv_tau;
            const float inner = is ? inner_is : mubar[j] - p_all;
            const float carry = has_next ? (is ? carry_is : abar[j]) : 0.0f;
            abar[j] = __builtin_fmaf(m_t, inner, carry);
        }
    }
}

} // namespace roi
