// wide.hip -- gfx950 kernels for groups of m = 16 and 32 weights.
//
// Four consecutive elements per lane (one Philox call, one 16-byte logits load
// and one 8-byte bf16 load per lane), a group spread over L = m / 4 adjacent
// lanes of one wave.  Group-wide maxima and "sum over the other lanes" use
// cross-lane butterflies: DPP quad permutations for lane distances 1..3 and
// the DPP half-row mirror for distances 4..7.  Every group is whole inside a wave and either
// all its lanes are active or none is, so the butterflies never read a lane
// outside the group.  Same arithmetic as the per-lane kernels for m = 4 and 8:
// the noise of noise.hpp, ranks with ties to the lower index, and the
// relaxation of relax.hpp in its "all entries but j" form.
#include <hip/hip_runtime.h>

#include <utility>

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
    const float span = (kmax - group_min<L>(min4(kappa))) * c;
    if (span <= exp_span) { // the same on all lanes of the group
        float ex[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) ex[e] = __builtin_amdgcn_exp2f(b[e] - bmax0);
#pragma unroll
        for (int k = 0; k < N; ++k) {
            float others[4], t;
            sums_but_one<4>(ex, others, t);
            const float ext = sum_other_lanes<L>(t);
            const float inv_total = __builtin_amdgcn_rcpf(t + ext);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float mu = ex[e] * inv_total;
                const float om = (others[e] + ext) * inv_total;
                if (want_s) S[e] += mu;
                if (kKeep) {
                    rec[k].mu[e] = mu;
                    rec[k].om[e] = om;
                }
                if (k + 1 < N) ex[e] = mu * pow_q<kQ>(om, inv_tau);
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
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float mu = ex[e] * inv_total;
            const float om = (others[e] + ext) * inv_total;
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
                const float rinv = live ? __builtin_amdgcn_rcpf(om) : 0.0f;
                mubar = __builtin_fmaf(-abar[e], rinv, sbar[e]);
                a_in[e] = live ? abar[e] : 0.0f;
            }
            t[e] = rec[k].mu[e] * mubar;
        }
        float q[4], tl;
        sums_but_one<4>(t, q, tl);
        const float ext = sum_other_lanes<L>(tl);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float x = __builtin_fmaf(rec[k].om[e], sbar[e], -(q[e] + ext));
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
    const bool lam_one = lambda == 1.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float ng = neg_gumbel_from_word(w[e], tab);
        const float phi_bar = lam_one ? phi[e] : phi[e] / lambda;
        kappa[e] = phi_bar - ng;
    }
}

// Forward.  Without kRelax (the straight-through forward with neither the
// soft mask nor the soft output) the ranks come from the hardware-log keys,
// and a wave with any group closer than their margin recomputes the exact
// keys; with kRelax the exact keys are needed for the relaxation anyway.
// kQ: how the exp-domain recursion raises omega to 1 / tau (relax.hpp pow_q).
template <int M, int N, bool kRelax, int kQ>
__global__ __launch_bounds__(kBlock) void fwd_wide_kernel(FwdBatch a)
{
    constexpr int L = M / 4;
    __shared__ float2 tab[kLogCells];
    fill_log_table(tab);
    __syncthreads();
    const FwdPiece& pc = a.p[find_piece(a)];
    NoiseKey key = a.key_base;
    key.block_hi = pc.block_hi;
    const int64_t nslots = pc.ngroups * L;
    const int64_t stride = (int64_t)pc.nblocks * kBlock;
    for (int64_t slot = (int64_t)(blockIdx.x - pc.first_block) * kBlock + threadIdx.x;
         slot < nslots; slot += stride) {
        const int part = (int)(slot % L);
        const int64_t group = slot / L;
        const f32x4 pv = stream_load(reinterpret_cast<const f32x4*>(pc.phi + slot * 4));
        const u32x2 wv = stream_load(reinterpret_cast<const u32x2*>(pc.W + slot * 4));
        const float phi[4] = {pv.x, pv.y, pv.z, pv.w};
        float kappa[4];
        bool keep[4];
        int sidx[4];
        bool decided = false;
        if constexpr (!kRelax) {
            const uint4 x = philox_block(pc.block0 + (uint32_t)slot, key);
            const float kf[4] = {fast_key_log2(phi[0], a.key_c, x.x),
                                 fast_key_log2(phi[1], a.key_c, x.y),
                                 fast_key_log2(phi[2], a.key_c, x.z),
                                 fast_key_log2(phi[3], a.key_c, x.w)};
            decided = __all(wide_top<L, N, false>(kf, part, keep, sidx));
        }
        if (!decided) {
            wide_keys(phi, pc.block0 + (uint32_t)slot, key, a.lambda, tab, kappa);
            wide_top<L, N, true>(kappa, part, keep, sidx);
        }
        const bool soft = kRelax && a.soft;
        if (!soft) {
            const uint32_t m01 = (keep[0] ? 0x0000FFFFu : 0u) | (keep[1] ? 0xFFFF0000u : 0u);
            const uint32_t m23 = (keep[2] ? 0x0000FFFFu : 0u) | (keep[3] ? 0xFFFF0000u : 0u);
            const u32x2 out = {wv.x & m01, wv.y & m23};
            stream_store(out, reinterpret_cast<u32x2*>(pc.Wm + slot * 4));
        }
        if (pc.idx) {
            // this lane holds ranks 4 part .. 4 part + 3
            uint8_t* dst = pc.idx + group * N + 4 * part;
            if (4 * part + 4 <= N) {
                const uint32_t w = (uint32_t)sidx[0] | ((uint32_t)sidx[1] << 8) |
                                   ((uint32_t)sidx[2] << 16) | ((uint32_t)sidx[3] << 24);
                if constexpr (N % 4 == 0)
                    stream_store(w, reinterpret_cast<uint32_t*>(dst));
                else
                    for (int e = 0; e < 4; ++e) dst[e] = (uint8_t)(w >> (8 * e));
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * part + e < N) dst[e] = (uint8_t)sidx[e];
            }
        }
        if constexpr (kRelax) {
            float S[4];
            StepRec<4> unused[N]; // not written when records are not kept
            wide_relax_forward<L, N, false, kQ>(kappa, kLog2e * a.inv_tau, a.inv_tau, a.exp_span,
                                                true, S, unused);
            if (pc.S) {
                const f32x4 sv = {S[0], S[1], S[2], S[3]};
                stream_store(sv, reinterpret_cast<f32x4*>(pc.S + slot * 4));
            }
            if (soft) { // pure soft forward: W (.) S, rounded to bf16
                const uint32_t h0 = float_to_bf16_rne(bf16_bits_to_float(wv.x & 0xFFFFu) * S[0]);
                const uint32_t h1 = float_to_bf16_rne(bf16_bits_to_float(wv.x >> 16) * S[1]);
                const uint32_t h2 = float_to_bf16_rne(bf16_bits_to_float(wv.y & 0xFFFFu) * S[2]);
                const uint32_t h3 = float_to_bf16_rne(bf16_bits_to_float(wv.y >> 16) * S[3]);
                const u32x2 out = {h0 | (h1 << 16), h2 | (h3 << 16)};
                stream_store(out, reinterpret_cast<u32x2*>(pc.Wm + slot * 4));
            }
        }
    }
}

// Backward; with kAdam the AdamW step on the logits is fused in (as in the
// per-lane kernels).
template <int M, int N, bool kAdam, int kQ>
__global__ __launch_bounds__(kBlock) void bwd_wide_kernel(BwdBatch a)
{
    constexpr int L = M / 4;
    const BwdPiece& pc = a.p[find_piece(a)];
    NoiseKey key = a.key_base;
    key.block_hi = pc.block_hi;
    const int64_t nslots = pc.ngroups * L;
    const int64_t stride = (int64_t)pc.nblocks * kBlock;
    for (int64_t slot = (int64_t)(blockIdx.x - pc.first_block) * kBlock + threadIdx.x;
         slot < nslots; slot += stride) {
        const f32x4 pv = stream_load(reinterpret_cast<const f32x4*>(pc.phi + slot * 4));
        const u32x2 wv = stream_load(reinterpret_cast<const u32x2*>(pc.W + slot * 4));
        const u32x2 gv = stream_load(reinterpret_cast<const u32x2*>(pc.G + slot * 4));
        f32x4 mv, vv;
        if constexpr (kAdam) {
            mv = stream_load(reinterpret_cast<const f32x4*>(pc.m + slot * 4));
            vv = stream_load(reinterpret_cast<const f32x4*>(pc.v + slot * 4));
        }
        float phi[4] = {pv.x, pv.y, pv.z, pv.w};
        // keys from the hardware logarithm, in log2 units (noise.hpp)
        const uint4 x = philox_block(pc.block0 + (uint32_t)slot, key);
        const float kappa[4] = {fast_key_log2(phi[0], a.key_c, x.x),
                                fast_key_log2(phi[1], a.key_c, x.y),
                                fast_key_log2(phi[2], a.key_c, x.z),
                                fast_key_log2(phi[3], a.key_c, x.w)};
        // Straight-through: dL/dS = dL/dW_masked (.) W, exact in fp32.
        const float sbar[4] = {
            bf16_bits_to_float(gv.x & 0xFFFFu) * bf16_bits_to_float(wv.x & 0xFFFFu),
            bf16_bits_to_float(gv.x >> 16) * bf16_bits_to_float(wv.x >> 16),
            bf16_bits_to_float(gv.y & 0xFFFFu) * bf16_bits_to_float(wv.y & 0xFFFFu),
            bf16_bits_to_float(gv.y >> 16) * bf16_bits_to_float(wv.y >> 16)};
        StepRec<4> rec[N];
        float S_unused[4];
        const bool exp_domain = wide_relax_forward<L, N, true, kQ>(
            kappa, a.inv_tau, a.inv_tau, a.exp_span, false, S_unused, rec);
        float abar[4];
        // Where every group of the wave took the exp-domain recursion, no
        // floor was reached and the sweep drops its selects (the two forms give
        // the same bits there, so this choice may be the wave's).  At m = 32
        // a second copy of the sweep would cost a wave per SIMD in registers.
        if (L <= 4 && __all(exp_domain))
            wide_relax_backward<L, N, kQ == 1, false>(rec, sbar, a.inv_tau, abar);
        else
            wide_relax_backward<L, N, kQ == 1, true>(rec, sbar, a.inv_tau, abar);
        // dL/dphi = dL/dkappa / lambda (the product is exact for lambda = 1)
        const float grad[4] = {abar[0] * a.inv_lambda, abar[1] * a.inv_lambda,
                               abar[2] * a.inv_lambda, abar[3] * a.inv_lambda};
        if (!kAdam || pc.dphi) store_f32<4>(pc.dphi + slot * 4, grad);
        if constexpr (kAdam) {
            float mo[4] = {mv.x, mv.y, mv.z, mv.w}, se[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) adamw_update(a.adam, grad[e], phi[e], mo[e], se[e]);
            store_f32<4>(const_cast<float*>(pc.phi) + slot * 4, phi);
            store_f32<4>(pc.m + slot * 4, mo);
            store_f32<4>(pc.v + slot * 4, se);
        }
    }
}

template <int M, int N>
FwdFn wide_fwd_q(bool relax, int q)
{
    if (!relax) return fwd_wide_kernel<M, N, false, 0>; // no relaxation
    return q == 1 ? fwd_wide_kernel<M, N, true, 1>
                  : (q == 2 ? fwd_wide_kernel<M, N, true, 2> : fwd_wide_kernel<M, N, true, 0>);
}

template <int M, int N, bool A>
BwdFn wide_bwd_q(int q)
{
    return q == 1 ? bwd_wide_kernel<M, N, A, 1>
                  : (q == 2 ? bwd_wide_kernel<M, N, A, 2> : bwd_wide_kernel<M, N, A, 0>);
}

template <int M, int... Ns>
FwdFn wide_fwd_for_n(int n, bool relax, int q, std::integer_sequence<int, Ns...>)
{
    FwdFn f = nullptr;
    ((n == Ns + 1 ? (f = wide_fwd_q<M, Ns + 1>(relax, q), 0) : 0), ...);
    return f;
}

template <int M, int... Ns>
BwdFn wide_bwd_for_n(int n, bool adam, int q, std::integer_sequence<int, Ns...>)
{
    BwdFn f = nullptr;
    ((n == Ns + 1 ? (f = adam ? wide_bwd_q<M, Ns + 1, true>(q) : wide_bwd_q<M, Ns + 1, false>(q), 0)
                  : 0),
     ...);
    return f;
}

} // namespace

FwdFn select_wide_fwd(int m, int n, bool relax, int q)
{
    if (m == 16) return wide_fwd_for_n<16>(n, relax, q, std::make_integer_sequence<int, 16>{});
    if (m == 32) return wide_fwd_for_n<32>(n, relax, q, std::make_integer_sequence<int, 32>{});
    return nullptr;
}

BwdFn select_wide_bwd(int m, int n, bool adam, int q)
{
    if (m == 16) return wide_bwd_for_n<16>(n, adam, q, std::make_integer_sequence<int, 16>{});
    if (m == 32) return wide_bwd_for_n<32>(n, adam, q, std::make_integer_sequence<int, 32>{});
    return nullptr;
}

} // namespace roi
