// wide.hpp -- device helpers of the gfx950 kernels for groups of m = 16 and 32
// weights (wide_fwd.hip, wide_bwd.hip), and of the backward for m = 8.
//
// Four consecutive elements per lane (one Philox call, one 16-byte logits load
// and one 8-byte bf16 load per lane), a group spread over L = m / 4 adjacent
// lanes of one wave.  Group-wide maxima and "sum over the other lanes" use
// cross-lane butterflies: DPP quad permutations for lane distances 1..3 and
// the DPP half-row mirror for distances 4..7.  Every group is whole inside a
// wave and either all its lanes are active or none is, so the butterflies
// never read a lane outside the group.  Same arithmetic as the per-lane
// kernels: the noise of noise.hpp, ranks with ties to the lower index, and the
// relaxation of relax.hpp in its "all entries but j" form.
#pragma once

#include <hip/hip_runtime.h>

#include "common.hpp"
#include "noise.hpp"
#include "relax.hpp"

namespace roi {
namespace {


// Value held by lane (lane ^ D) of the same group (D < 8), with DPP only:
// quad permutations for D < 4; for D >= 4, the half-row mirror (lane i of an
// 8-lane half to lane 7 - i, i.e. xor 7) followed by the quad permutation of
// D ^ 7.
template <int D>
__device__ __forceinline__ float lane_xor(float v)
{
    static_assert(D > 0 && D < 8, "lane distance");
    int x = __float_as_int(v);
    if constexpr ((D & 4) != 0) x = __builtin_amdgcn_update_dpp(0, x, 0x141, 0xF, 0xF, true);
    constexpr int lo = ((D & 4) != 0 ? (D ^ 7) : D) & 3;
    if constexpr (lo == 1) x = __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, true); // [1,0,3,2]
    if constexpr (lo == 2) x = __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, true); // [2,3,0,1]
    if constexpr (lo == 3) x = __builtin_amdgcn_update_dpp(0, x, 0x1B, 0xF, 0xF, true); // [3,2,1,0]
    return __int_as_float(x);
}

template <int L>
__device__ __forceinline__ float group_max(float v)
{
    v = fmaxf(v, lane_xor<1>(v));
    if constexpr (L >= 4) v = fmaxf(v, lane_xor<2>(v));
    if constexpr (L >= 8) v = fmaxf(v, lane_xor<4>(v));
    return v;
}

// Sum of t over the other L - 1 lanes of the group (never includes this lane's
// own t, so a dominant lane does not swamp the others).
template <int L>
__device__ __forceinline__ float sum_other_lanes(float t)
{
    const float o1 = lane_xor<1>(t);
    if constexpr (L == 2) return o1;
    const float s1 = t + o1; // pair sum
    float other = o1 + lane_xor<2>(s1);
    if constexpr (L == 8) {
        const float s2 = s1 + lane_xor<2>(s1); // quad sum
        other += lane_xor<4>(s2);
    }
    return other;
}

__device__ __forceinline__ float max4(const float (&x)[4])
{
    return fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
}

template <int L>
__device__ __forceinline__ float group_min(float v)
{
    v = fminf(v, lane_xor<1>(v));
    if constexpr (L >= 4) v = fminf(v, lane_xor<2>(v));
    if constexpr (L >= 8) v = fminf(v, lane_xor<4>(v));
    return v;
}

__device__ __forceinline__ float min4(const float (&x)[4])
{
    return fminf(fminf(x[0], x[1]), fminf(x[2], x[3]));
}

// Hard top-n by a bitonic sort of the group (descending), entry i = 4 part + e
// of the group at lane `part`, slot e.  Each key travels with its index.  An
// entry beats another when its key is larger, or (kTies) equal with a lower
// index: the order of the ranks, ties to the lower index.  Without kTies the
// keys must be distinct for the result to mean anything (the caller checks).
// A stage (kk, j) pairs entry i with i ^ j; the pair is ordered descending
// when (i & kk) == 0 and ascending otherwise, the lower entry of a
// descending pair keeping the entry that beats.  j = 1, 2 pair slots of one
// lane; j >= 4 pairs lane part with lane part ^ (j / 4), each lane keeping
// one side of its four pairs.  The network is log2(m) (log2(m) + 1) / 2
// stages of 4 entries per lane, against m comparisons per entry for counting
// ranks, and keeps few values live.
template <bool kTies>
__device__ __forceinline__ bool beats(float ka, int ia, float kb, int ib)
{
    return kTies ? (ka > kb || (ka == kb && ia < ib)) : ka > kb;
}

template <int KK, int J, bool kTies>
__device__ __forceinline__ void bitonic_stage(float (&k)[4], int (&ix)[4], int part)
{
    if constexpr (J < 4) {
#pragma unroll
        for (int lo = 0; lo < 4; ++lo) {
            if ((lo & J) != 0) continue;
            const int hi = lo | J;
            // direction of the pair: (i & KK) with i = 4 part + lo
            const bool desc = KK < 4 ? ((lo & KK) == 0) : ((part & (KK >> 2)) == 0);
            const bool sw = beats<kTies>(k[hi], ix[hi], k[lo], ix[lo]) == desc;
            const float kl = k[lo], kh = k[hi];
            const int il = ix[lo], ih = ix[hi];
            k[lo] = sw ? kh : kl;
            k[hi] = sw ? kl : kh;
            ix[lo] = sw ? ih : il;
            ix[hi] = sw ? il : ih;
        }
    } else {
        constexpr int D = J / 4; // lane distance
        const bool lower = (part & D) == 0;
        const bool desc = (part & (KK >> 2)) == 0;
        const bool keep_max = lower == desc;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float o = lane_xor<D>(k[e]);
            const int oi = __float_as_int(lane_xor<D>(__int_as_float(ix[e])));
            const bool take = beats<kTies>(o, oi, k[e], ix[e]) == keep_max;
            k[e] = take ? o : k[e];
            ix[e] = take ? oi : ix[e];
        }
    }
}

template <int M, int KK, int J, bool kTies>
__device__ __forceinline__ void bitonic_from(float (&k)[4], int (&ix)[4], int part)
{
    bitonic_stage<KK, J, kTies>(k, ix, part);
    if constexpr (J > 1)
        bitonic_from<M, KK, J / 2, kTies>(k, ix, part);
    else if constexpr (KK < M)
        bitonic_from<M, KK * 2, KK, kTies>(k, ix, part);
}

// Sorts the group's keys (four per lane, kf) and sets keep[e] (is this lane's
// entry e among the n that beat the others) and sidx[e] (the index within the
// group of the entry at sorted position 4 part + e, i.e. of rank 4 part + e).
// For the hardware-log keys (kTies false) it returns whether every two keys of
// the group are further apart than the margin of their errors (noise.hpp):
// then the order is the exact keys' order and no two tie, and checking the
// m - 1 pairs adjacent in the sorted order covers every pair.  For exact keys
// (kTies) ties go to the lower index and the return value is true.
template <int L, int N, bool kTies>
__device__ __forceinline__ bool wide_top(const float (&kf)[4], int part, bool (&keep)[4],
                                         int (&sidx)[4])
{
    constexpr int M = 4 * L;
    float k[4] = {kf[0], kf[1], kf[2], kf[3]};
#pragma unroll
    for (int e = 0; e < 4; ++e) sidx[e] = 4 * part + e;
    bitonic_from<M, 2, 1, kTies>(k, sidx, part);
    const int lane = (int)(threadIdx.x & 63);
    // the entry of rank n - 1, held by lane (n - 1) / 4 of the group
    const int src = lane - part + (N - 1) / 4;
    const float kth = __shfl(k[(N - 1) % 4], src);
    const int ith = __shfl(sidx[(N - 1) % 4], src);
#pragma unroll
    for (int e = 0; e < 4; ++e)
        keep[e] = kTies ? !beats<true>(kth, ith, kf[e], 4 * part + e) : kf[e] >= kth;
    if constexpr (kTies) return true;
    float big = fmaxf(fmaxf(fabsf(kf[0]), fabsf(kf[1])), fmaxf(fabsf(kf[2]), fabsf(kf[3])));
    big = group_max<L>(big);
    const float margin = __builtin_fmaf(big, 0x1p-20f, kFastPairMargin);
    // adjacent sorted pairs: three in the lane, and the lane's last with the
    // next lane's first (the group's last lane has no successor)
    bool sep = (k[0] - k[1] > margin) & (k[1] - k[2] > margin) & (k[2] - k[3] > margin);
    const float next = __shfl(k[0], part + 1 < L ? lane + 1 : lane);
    sep &= (part + 1 == L) || (k[3] - next > margin);
    return sep;
}

// Relaxation over the group (§3.2 recursion, Algorithm 1), four entries per
// lane: the exp-domain recursion of relax_forward_exp when the group's key
// span is at most exp_span (the host's bound, relax.hpp), else the log-domain
// loop of relax_forward, with sums over the group's other lanes.  The choice
// is the group's own (all its lanes agree), so its outputs do not depend on
// which groups share its wave.  Returns true when this group took the
// exp-domain path (its omegas then never reach the floor).
template <int L, int N, bool kKeep, int kQ>
__device__ __forceinline__ bool wide_relax_forward(const float (&kappa)[4], float key_scale,
                                                   float inv_tau, float exp_span, bool want_s,
                                                   float (&S)[4], StepRec<4> (&rec)[N])
{
    // b = kappa * key_scale unshifted, each step subtracting its own largest b
    // (see scaled_keys in relax.hpp)
    const float kmax = group_max<L>(max4(kappa));
    const float c = key_scale;
    const float bmax0 = kmax * c;
    float b[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        b[e] = kappa[e] * c;
        S[e] = 0.0f;
    }
    // kQ < 0: the exp-domain form is off at this temperature (no span needed)
    const float span = kQ < 0 ? 0.0f : (kmax - group_min<L>(min4(kappa))) * c;
    if (kQ >= 0 && span <= exp_span) { // the same on all lanes of the group
        float ex[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) ex[e] = __builtin_amdgcn_exp2f(b[e] - bmax0);
#pragma unroll
        for (int k = 0; k < N; ++k) {
            float others[4], t;
            sums_but_one<4>(ex, others, t);
            const float ext = sum_other_lanes<L>(t);
            const float inv_total = __builtin_amdgcn_rcpf(t + ext);
            const float ext_w = ext * inv_total; // the other lanes' weight
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float mu = ex[e] * inv_total;
                const float om = __builtin_fmaf(others[e], inv_total, ext_w);
                if (want_s) S[e] += mu;
                if (kKeep) {
                    rec[k].mu[e] = mu;
                    rec[k].om[e] = om;
                }
                if (k + 1 < N) ex[e] = mu * pow_q<kQ < 0 ? 0 : kQ>(om, inv_tau);
            }
        }
        return true;
    }
#pragma unroll
    for (int k = 0; k < N; ++k) {
        float ex[4];
        const float bmax = k == 0 ? bmax0 : group_max<L>(max4(b));
#pragma unroll
        for (int e = 0; e < 4; ++e) ex[e] = __builtin_amdgcn_exp2f(b[e] - bmax);
        float others[4], t;
        sums_but_one<4>(ex, others, t);
        const float ext = sum_other_lanes<L>(t);
        const float inv_total = __builtin_amdgcn_rcpf(t + ext);
        const float ext_w = ext * inv_total; // the other lanes' weight
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float mu = ex[e] * inv_total;
            const float om = __builtin_fmaf(others[e], inv_total, ext_w);
            if (want_s) S[e] += mu;
            if (kKeep) {
                rec[k].mu[e] = mu;
                rec[k].om[e] = om;
            }
            if (k + 1 < N)
                b[e] = __builtin_fmaf(__builtin_amdgcn_logf(fmaxf(om, kFltMin)), inv_tau, b[e]);
        }
    }
    return false;
}

// Reverse sweep over the group: relax_backward of relax.hpp (one form for
// every entry; with kFloor, floored logs pass no derivative), with the sum over
// the other entries taken across the group's lanes.
template <int L, int N, bool kTauIsOne, bool kFloor>
__device__ __forceinline__ void wide_relax_backward(const StepRec<4> (&rec)[N],
                                                    const float (&sbar)[4], float inv_tau,
                                                    float (&abar)[4])
{
#pragma unroll
    for (int k = N - 1; k >= 0; --k) {
        const bool has_next = (k + 1 < N);
        float t[4], a_in[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float mubar = sbar[e];
            a_in[e] = 0.0f;
            if (has_next) {
                const float om = rec[k].om[e];
                const bool live = !kFloor || om >= kFltMin;
                // 1/inf = 0 for a floored entry.  Selecting the reciprocal's
                // input, not its result, leaves the two copies of the sweep
                // (with and without the selects) no reciprocal in common, so
                // the compiler does not compute them ahead of the choice and
                // hold them in registers beside the records.
                const float rinv = __builtin_amdgcn_rcpf(live ? om : __builtin_inff());
                mubar = __builtin_fmaf(-abar[e], rinv, sbar[e]);
                a_in[e] = live ? abar[e] : 0.0f;
            }
            t[e] = rec[k].mu[e] * mubar;
        }
        // Sum over the group's entries but e: the other lanes' sum enters the
        // two pair sums of this lane, so each is one add from them (no
        // subtraction).
        const float pa = t[0] + t[1], pb = t[2] + t[3];
        const float ext = sum_other_lanes<L>(pa + pb);
        const float pae = pa + ext, pbe = pb + ext;
        const float q[4] = {t[1] + pbe, t[0] + pbe, pae + t[3], pae + t[2]};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float x = __builtin_fmaf(rec[k].om[e], sbar[e], -q[e]);
            const float m_t = kTauIsOne ? rec[k].mu[e] : rec[k].mu[e] * inv_tau;
            abar[e] = has_next ? __builtin_fmaf(m_t, x - a_in[e], abar[e]) : m_t * x;
        }
    }
}

__device__ __forceinline__ void wide_keys(const float (&phi)[4], uint32_t block, const NoiseKey& key,
                                          float lambda, const float2* tab, float (&kappa)[4])
{
    const uint4 x = philox_block(block, key);
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
    float phi_bar[4];
    scaled_logits4(phi, lambda, phi_bar);
#pragma unroll
    for (int e = 0; e < 4; ++e) kappa[e] = phi_bar[e] - neg_gumbel_from_word(w[e], tab);
}

} // namespace
} // namespace roi
