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

// Backward; with kAdam the AdamW step on the logits is fused in (as in the
// per-lane kernels).
template <int M, int N, bool kAdam, int kQ>
__global__ __launch_bounds__(kBlock) void bwd_wide_kernel(BwdBatch a)
{
    constexpr int L = M / 4;
    // A select-free copy of the sweep beside the one with floor selects.  At
    // m = 32 the kernel holds about 28 + 8n VGPRs (8 per step of records) and
    // the second copy 8 more; at tau != 1 or with AdamW it needs far more.
    // It is taken where it costs no wave per SIMD.
    constexpr bool kTwoSweeps =
        L <= 4 || (kQ == 1 && !kAdam && waves_for_vgprs(36 + 8 * N) == waves_for_vgprs(28 + 8 * N));
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
        // the same bits there, so this choice may be the wave's).
        if (kTwoSweeps && __all(exp_domain))
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

template <int M, int N, bool A>
BwdFn wide_bwd_q(int q)
{
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

BwdFn select_wide_bwd(int m, int n, bool adam, int q)
{
    if (m == 8) return wide_bwd_for_n<8>(n, adam, q, std::make_integer_sequence<int, 8>{});
    if (m == 16) return wide_bwd_for_n<16>(n, adam, q, std::make_integer_sequence<int, 16>{});
    if (m == 32) return wide_bwd_for_n<32>(n, adam, q, std::make_integer_sequence<int, 32>{});
    return nullptr;
}

} // namespace roi
