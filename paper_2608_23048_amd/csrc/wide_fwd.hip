// wide_fwd.hip -- the forward kernel for groups of m = 16 and 32 weights
// (helpers and layout in wide.hpp).
#include <hip/hip_runtime.h>

#include <utility>

#include "wide.hpp"

namespace roi {
namespace {

// Forward.  Without kRelax (the straight-through forward with neither the
// soft mask nor the soft output) the ranks come from the hardware-log keys,
// and a wave with any group closer than their margin recomputes the exact
// keys; with kRelax the exact keys are needed for the relaxation anyway.
// kQ: how the exp-domain recursion raises omega to 1 / tau (relax.hpp pow_q).
template <int M, int N, bool kRelax, int kQ>
__global__ __launch_bounds__(kBlock) void fwd_wide_kernel(FwdBatch a)
{
    constexpr int L = M / 4;
    // The exact keys read the log cells: from LDS when every group needs them
    // (kRelax), else (only groups of waves with near ties) from global memory,
    // where they stay cached, so that a block starts without a barrier.
    __shared__ float2 tab_lds[kRelax ? kLogCells : 1];
    const float2* tab = kRelax ? tab_lds : kLogCellTable.cell;
    if constexpr (kRelax) {
        fill_log_table(tab_lds);
        __syncthreads();
    }
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
            wide_relax_forward<L, N, false, kQ>(kappa, a.key_scale, a.inv_tau, a.exp_span,
                                                true, S, unused);
            if (pc.S) {
                const f32x4 sv = {S[0], S[1], S[2], S[3]};
                stream_store(sv, reinterpret_cast<f32x4*>(pc.S + slot * 4));
            }
            if (soft) // pure soft forward: W (.) S, rounded to bf16
                stream_store(soft_product4(wv.x, wv.y, S), reinterpret_cast<u32x2*>(pc.Wm + slot * 4));
        }
    }
}

// One slot of the pure soft forward: the loads go out first, the slot's noise
// is computed while they are in flight, and a kFull pass has no per-lane
// condition (as the backward's spans, wide_bwd.hip).
template <int M, int N, int kQ, bool kFull>
__device__ __forceinline__ void soft_wide_slot(const FwdBatch& a, const FwdPiece& pc,
                                               const NoiseKey& key, float2* tab, int64_t slot,
                                               int64_t nslots)
{
    constexpr int L = M / 4;
    const float4 cells = log_cells_of_lane();
    __builtin_amdgcn_sched_barrier(0);
    f32x4 pv{};
    u32x2 wv{};
    if (kFull || slot < nslots) {
        pv = stream_load(reinterpret_cast<const f32x4*>(pc.phi + slot * 4));
        wv = stream_load(reinterpret_cast<const u32x2*>(pc.W + slot * 4));
    }
    __builtin_amdgcn_sched_barrier(0);
    float ng[4];
    {
        const uint4 x = philox_block(pc.block0 + (uint32_t)slot, key);
        const uint32_t w[4] = {x.x, x.y, x.z, x.w};
        publish_log_table(tab, cells);
#pragma unroll
        for (int e = 0; e < 4; ++e) ng[e] = neg_gumbel_from_word(w[e], tab);
    }
    __builtin_amdgcn_sched_barrier(0);
    // a group's lanes are all live or all past the end (groups are whole in a wave)
    if (!kFull && slot >= nslots) return;
    const float phi[4] = {pv.x, pv.y, pv.z, pv.w};
    float kappa[4];
    scaled_logits4(phi, a.lambda, kappa);
#pragma unroll
    for (int e = 0; e < 4; ++e) kappa[e] -= ng[e];
    float S[4];
    StepRec<4> unused[N]; // not written when records are not kept
    wide_relax_forward<L, N, false, kQ>(kappa, a.key_scale, a.inv_tau, a.exp_span, true, S,
                                        unused);
    stream_store(soft_product4(wv.x, wv.y, S), reinterpret_cast<u32x2*>(pc.Wm + slot * 4));
}

// Pure soft forward whose only output is bf16(W (.) S): the relaxation at the
// exact keys, no selection.  The block's waves share one copy of the log
// cells in LDS (noise.hpp), so a block starts streaming without a barrier.
template <int M, int N, int kQ>
__global__ __launch_bounds__(kBlock) void fwd_soft_wide_kernel(FwdBatch a)
{
    __shared__ float4 tab4[kLogCells / 2];
    float2* tab = reinterpret_cast<float2*>(tab4);
    const FwdPiece& pc = a.p[find_piece(a)];
    NoiseKey key = a.key_base;
    key.block_hi = pc.block_hi;
    const int64_t nslots = pc.ngroups * (M / 4);
    const int64_t stride = (int64_t)pc.nblocks * kBlock;
    for (int64_t base = (int64_t)(blockIdx.x - pc.first_block) * kBlock; base < nslots;
         base += stride) {
        if (base + kBlock <= nslots)
            soft_wide_slot<M, N, kQ, true>(a, pc, key, tab, base + threadIdx.x, nslots);
        else
            soft_wide_slot<M, N, kQ, false>(a, pc, key, tab, base + threadIdx.x, nslots);
    }
}

template <int M, int N>
FwdFn wide_soft_q(int q)
{
    if (q < 0) return fwd_soft_wide_kernel<M, N, -1>;
    return q == 1 ? fwd_soft_wide_kernel<M, N, 1>
                  : (q == 2 ? fwd_soft_wide_kernel<M, N, 2> : fwd_soft_wide_kernel<M, N, 0>);
}

template <int M, int... Ns>
FwdFn wide_soft_for_n(int n, int q, std::integer_sequence<int, Ns...>)
{
    FwdFn f = nullptr;
    ((n == Ns + 1 ? (f = wide_soft_q<M, Ns + 1>(q), 0) : 0), ...);
    return f;
}

template <int M, int N>
FwdFn wide_fwd_q(bool relax, int q)
{
    if (!relax) return fwd_wide_kernel<M, N, false, 0>; // no relaxation
    return q == 1 ? fwd_wide_kernel<M, N, true, 1>
                  : (q == 2 ? fwd_wide_kernel<M, N, true, 2> : fwd_wide_kernel<M, N, true, 0>);
}

template <int M, int... Ns>
FwdFn wide_fwd_for_n(int n, bool relax, int q, std::integer_sequence<int, Ns...>)
{
    FwdFn f = nullptr;
    ((n == Ns + 1 ? (f = wide_fwd_q<M, Ns + 1>(relax, q), 0) : 0), ...);
    return f;
}

} // namespace

FwdFn select_wide_soft_only(int m, int n, int q)
{
    if (m == 16) return wide_soft_for_n<16>(n, q, std::make_integer_sequence<int, 16>{});
    if (m == 32) return wide_soft_for_n<32>(n, q, std::make_integer_sequence<int, 32>{});
    return nullptr;
}

FwdFn select_wide_fwd(int m, int n, bool relax, int q)
{
    if (m == 16) return wide_fwd_for_n<16>(n, relax, q, std::make_integer_sequence<int, 16>{});
    if (m == 32) return wide_fwd_for_n<32>(n, relax, q, std::make_integer_sequence<int, 32>{});
    return nullptr;
}

} // namespace roi
