// wide_bwd.hip -- the backward kernel (optionally with the fused AdamW step)
// for groups of m = 8, 16 and 32 weights (helpers and layout in wide.hpp).
// At m = 8 a group spans two lanes: half the relaxation records per lane of
// the one-group-per-lane layout, so twice the waves per SIMD.
#include <hip/hip_runtime.h>

#include <utility>

#include "wide.hpp"

namespace roi {
namespace {

// Waves per SIMD of a kernel of v VGPRs (512 per SIMD lane, allocated in
// blocks of 8, at most 8 waves).
constexpr int waves_for_vgprs(int v)
{
    const int w = 512 / ((v + 7) / 8 * 8);
    return w < 8 ? w : 8;
}

// Chunks of kBlock slots a block walks, loading the next chunk while it
// computes one.  One for every m: the wide kernels hold many relaxation
// records per lane, and a second set of inputs and noise costs them waves
// per SIMD (4:8 went from 6 to 4).
#ifndef ROI_WIDE_BWD_CHUNKS_M8
#define ROI_WIDE_BWD_CHUNKS_M8 1
#endif
template <int M>
constexpr int kWideBwdChunks = M == 8 ? ROI_WIDE_BWD_CHUNKS_M8 : 1;

// The backward of one slot (four consecutive elements of a group of m, the
// group spread over m / 4 adjacent lanes) given its noise ng = -g; with kAdam
// the AdamW step on the logits is fused in (as in the per-lane kernels).
template <int M, int N, bool kAdam, int kQ>
__device__ __forceinline__ void bwd_wide_slot(const BwdBatch& a, const BwdPiece& pc,
                                              const float (&ng)[4], const BwdSlot<kAdam>& in,
                                              int64_t slot)
{
    constexpr int L = M / 4;
    // A select-free copy of the sweep beside the one with floor selects.  At
    // m = 32 the kernel holds about 28 + 8n VGPRs (8 per step of records) and
    // the second copy 8 more; at tau != 1 or with AdamW it needs far more.
    // It is taken where it costs no wave per SIMD.
    constexpr bool kTwoSweeps =
        kQ >= 0 &&
        (L <= 4 || (kQ == 1 && !kAdam && waves_for_vgprs(36 + 8 * N) == waves_for_vgprs(28 + 8 * N)));
    float phi[4] = {in.phi.x, in.phi.y, in.phi.z, in.phi.w};
    // the keys the forward sampled: kappa = fl(fl(phi / lambda) + g) (noise.hpp)
    float kappa[4];
    scaled_logits4(phi, a.lambda, kappa);
#pragma unroll
    for (int e = 0; e < 4; ++e) kappa[e] -= ng[e];
    // Straight-through: dL/dS = dL/dW_masked (.) W, exact in fp32.
    const float sbar[4] = {
        bf16_bits_to_float(in.g.x & 0xFFFFu) * bf16_bits_to_float(in.w.x & 0xFFFFu),
        bf16_bits_to_float(in.g.x >> 16) * bf16_bits_to_float(in.w.x >> 16),
        bf16_bits_to_float(in.g.y & 0xFFFFu) * bf16_bits_to_float(in.w.y & 0xFFFFu),
        bf16_bits_to_float(in.g.y >> 16) * bf16_bits_to_float(in.w.y >> 16)};
    StepRec<4> rec[N];
    float S_unused[4];
    const bool exp_domain = wide_relax_forward<L, N, true, kQ>(
        kappa, a.key_scale, a.inv_tau, a.exp_span, false, S_unused, rec);
    float abar[4];
    // Where every group of the wave took the exp-domain recursion, no floor
    // was reached and the sweep drops its selects (the two forms give the same
    // bits there, so this choice may be the wave's).
    if (kTwoSweeps && __all(exp_domain))
        wide_relax_backward<L, N, kQ == 1, false>(rec, sbar, a.inv_tau, abar);
    else
        wide_relax_backward<L, N, kQ == 1, true>(rec, sbar, a.inv_tau, abar);
    // dL/dphi = dL/dkappa / lambda (the product is exact for lambda = 1)
    const float grad[4] = {abar[0] * a.inv_lambda, abar[1] * a.inv_lambda, abar[2] * a.inv_lambda,
                           abar[3] * a.inv_lambda};
    if (!kAdam || pc.dphi) store_f32<4>(pc.dphi + slot * 4, grad);
    if constexpr (kAdam) {
        float mo[4] = {in.mom.x, in.mom.y, in.mom.z, in.mom.w};
        float se[4] = {in.sec.x, in.sec.y, in.sec.z, in.sec.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) adamw_update(a.adam, grad[e], phi[e], mo[e], se[e]);
        store_f32<4>(const_cast<float*>(pc.phi) + slot * 4, phi);
        store_f32<4>(pc.m + slot * 4, mo);
        store_f32<4>(pc.v + slot * 4, se);
    }
}

// The noise of a slot's four elements (one Philox block), ng = -g.
__device__ __forceinline__ void slot_noise(uint32_t block, const NoiseKey& key, const float2* tab,
                                           float (&ng)[4])
{
    const uint4 x = philox_block(block, key);
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) ng[e] = neg_gumbel_from_word(w[e], tab);
}

// kWideBwdChunks<M> chunks of kBlock slots from `base`, as the per-lane
// backward walks its chunks (roi.hip): the loads go out first, each chunk's
// noise runs while loads are in flight, and kFull spans have no per-lane
// condition.  A group's lanes are all inside the piece or all past it.
template <int M, int N, bool kAdam, int kQ, bool kFull>
__device__ __forceinline__ void bwd_wide_span(const BwdBatch& a, const BwdPiece& pc,
                                              const NoiseKey& key, float2* tab, int64_t base,
                                              int64_t nslots)
{
    constexpr int K = kWideBwdChunks<M>;
    const int64_t s0 = base + threadIdx.x;
    BwdSlot<kAdam> in[2];
    if (kFull || s0 < nslots) load_bwd_slot<kAdam>(pc, s0, in[0]);
    __builtin_amdgcn_sched_barrier(0);
    const float4 cells = log_cells_of_lane();
    __builtin_amdgcn_sched_barrier(0);
    if (K > 1 && (kFull || s0 + kBlock < nslots)) load_bwd_slot<kAdam>(pc, s0 + kBlock, in[1]);
    __builtin_amdgcn_sched_barrier(0);
    float ng[2][4];
    {
        const uint4 x = philox_block(pc.block0 + (uint32_t)s0, key);
        const uint32_t w[4] = {x.x, x.y, x.z, x.w};
        publish_log_table(tab, cells);
#pragma unroll
        for (int e = 0; e < 4; ++e) ng[0][e] = neg_gumbel_from_word(w[e], tab);
    }
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int64_t s = s0 + (int64_t)k * kBlock;
        if (k + 1 < K) slot_noise(pc.block0 + (uint32_t)(s + kBlock), key, tab, ng[(k + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
        if (kFull || s < nslots) bwd_wide_slot<M, N, kAdam, kQ>(a, pc, ng[k & 1], in[k & 1], s);
        if (k + 2 < K && (kFull || s + 2 * kBlock < nslots))
            load_bwd_slot<kAdam>(pc, s + 2 * kBlock, in[k & 1]);
    }
}

// Backward; with kAdam the AdamW step on the logits is fused in.  Every group
// takes the exact keys; the block's waves share one copy of the log cells in
// LDS (noise.hpp).
template <int M, int N, bool kAdam, int kQ>
__global__ __launch_bounds__(kBlock) void bwd_wide_kernel(BwdBatch a)
{
    __shared__ float4 tab4[kLogCells / 2];
    float2* tab = reinterpret_cast<float2*>(tab4);
    const BwdPiece& pc = a.p[find_piece(a)];
    NoiseKey key = a.key_base;
    key.block_hi = pc.block_hi;
    const int64_t nslots = pc.ngroups * (M / 4);
    const int64_t span = (int64_t)kBlock * kWideBwdChunks<M>;
    for (int64_t base = (int64_t)(blockIdx.x - pc.first_block) * span; base < nslots;
         base += (int64_t)pc.nblocks * span) {
        if (base + span <= nslots)
            bwd_wide_span<M, N, kAdam, kQ, true>(a, pc, key, tab, base, nslots);
        else
            bwd_wide_span<M, N, kAdam, kQ, false>(a, pc, key, tab, base, nslots);
    }
}

template <int M, int N, bool A>
BwdFn wide_bwd_q(int q)
{
    if (q < 0) return bwd_wide_kernel<M, N, A, -1>;
    return q == 1 ? bwd_wide_kernel<M, N, A, 1>
                  : (q == 2 ? bwd_wide_kernel<M, N, A, 2> : bwd_wide_kernel<M, N, A, 0>);
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

int64_t wide_bwd_block_slots(int m)
{
    return (int64_t)kBlock * (m == 8 ? kWideBwdChunks<8> : 1);
}

BwdFn select_wide_bwd(int m, int n, bool adam, int q)
{
    if (m == 8) return wide_bwd_for_n<8>(n, adam, q, std::make_integer_sequence<int, 8>{});
    if (m == 16) return wide_bwd_for_n<16>(n, adam, q, std::make_integer_sequence<int, 16>{});
    if (m == 32) return wide_bwd_for_n<32>(n, adam, q, std::make_integer_sequence<int, 32>{});
    return nullptr;
}

} // namespace roi
