// roi.hip -- gfx950 kernels and the C ABI of the RoI N:M mask sampler.
//
// Work decomposition: one group of m consecutive weights per lane.  A wave of
// 64 lanes covers 64 consecutive groups, so each load and store instruction of
// a wave touches one contiguous span (64 * 16 B of logits, 64 * 2m B of bf16
// weights); blocks walk the tensor in a grid-stride loop.  Everything a group
// needs stays in registers: the Philox words, the keys, the ranks and, in the
// backward, the n softmax records of the relaxation.  The path is a stream of
// elementwise work with per-group reductions, so it is bound by HBM bandwidth
// or VALU issue, never by a dense contraction; there is no MFMA here.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <algorithm>
#include <utility>
#include <vector>

#include "common.hpp"
#include "host.hpp"
#include "noise.hpp"
#include "relax.hpp"
#include "roi.h"

// ----------------------------------------------------------------------------- host helpers
// (declared in host.hpp; shared by the translation units of the library; the
// argument checks themselves are in checks.cpp)
namespace roi {

// Grid for `items` work items of one thread each: one block per `block` items
// (a one-shot grid dispatched in address order keeps the set of DRAM pages in
// use compact; measured on MI355X, a plain copy streams at ~6.3 TB/s this way
// against ~5 TB/s with a fixed grid looping with a large stride).  A dispatch
// holds its total work-item count in 32 bits, so grids stop below 2^32
// threads; kernels keep a stride loop for the items beyond.
int grid_for(int64_t items, int block)
{
    const int64_t max_blocks = (int64_t)(0xFFFFFFFFu / (uint32_t)block);
    const int64_t need = (items + block - 1) / block;
    return (int)(need < 1 ? 1 : (need < max_blocks ? need : max_blocks));
}


NoiseKey make_key(uint64_t seed, uint64_t step, uint64_t block)
{
    NoiseKey k;
    k.k0 = (uint32_t)seed;
    k.k1 = (uint32_t)(seed >> 32);
    k.step_lo = (uint32_t)step;
    k.step_hi = (uint32_t)(step >> 32);
    k.block_hi = (uint32_t)(block >> 32);
    return k;
}

int launch_status(const char* what)
{
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(ROI_E_HIP, "%s: launch failed: %s", what, hipGetErrorString(e));
    return ok();
}

} // namespace roi

namespace roi {
namespace {

// Groups each lane of the forward loads ahead before computing the first, per
// m, and the block size of the per-lane kernels.
#ifndef ROI_UNROLL_FWD_M4
#define ROI_UNROLL_FWD_M4 2
#endif
#ifndef ROI_UNROLL_FWD_M8
#define ROI_UNROLL_FWD_M8 1
#endif

#ifndef ROI_LANE_BLOCK
#define ROI_LANE_BLOCK 256
#endif
#ifndef ROI_BWD_CHUNKS
#define ROI_BWD_CHUNKS 2
#endif
template <int M>
constexpr int kUnrollFwd = M == 4 ? ROI_UNROLL_FWD_M4 : ROI_UNROLL_FWD_M8;
constexpr int kBwdChunks = ROI_BWD_CHUNKS; // chunks per block in the m = 4 backward
constexpr int kLaneBlock = ROI_LANE_BLOCK;
static_assert(kLaneBlock >= kLogCells + 64 && kLaneBlock % 64 == 0, "lane block size");

// bf16(W (.) S) of one group, stored: w holds the bf16 patterns of W in
// pairs (load_bf16_pairs).
template <int M>
__device__ __forceinline__ void store_soft_product(uint16_t* p, const uint32_t (&w)[M / 2],
                                                   const float (&S)[M])
{
#pragma unroll
    for (int t = 0; t < M / 4; ++t)
        stream_store(soft_product4(w[2 * t], w[2 * t + 1], S + 4 * t),
                     reinterpret_cast<u32x2*>(p) + t);
}

// Masked bf16 weights: the kept value, or +0.0 (bits 0x0000).
template <int M>
__device__ __forceinline__ void store_masked(uint16_t* p, const uint32_t (&w)[M], const int (&rank)[M],
                                             int n)
{
    uint32_t packed[M / 2];
#pragma unroll
    for (int t = 0; t < M / 2; ++t) {
        const uint32_t lo = rank[2 * t] < n ? w[2 * t] : 0u;
        const uint32_t hi = rank[2 * t + 1] < n ? w[2 * t + 1] : 0u;
        packed[t] = lo | (hi << 16);
    }
    if constexpr (M == 4) {
        const u32x2 v = {packed[0], packed[1]};
        stream_store(v, reinterpret_cast<u32x2*>(p));
    } else {
        const u32x4 v = {packed[0], packed[1], packed[2], packed[3]};
        stream_store(v, reinterpret_cast<u32x4*>(p));
    }
}

// n index bytes of a group, already packed (byte r = index of rank r).
template <int N>
__device__ __forceinline__ void store_order(uint8_t* p, uint32_t packed)
{
    if constexpr (N == 1) {
        stream_store((uint8_t)packed, p);
    } else if constexpr (N == 2) {
        stream_store((uint16_t)packed, reinterpret_cast<uint16_t*>(p));
    } else if constexpr (N == 4) {
        stream_store(packed, reinterpret_cast<uint32_t*>(p));
    } else {
#pragma unroll
        for (int r = 0; r < N; ++r) p[r] = (uint8_t)(packed >> (8 * r));
    }
}

// Selected indices in selection order: byte r holds the index of rank r.
template <int N>
__device__ __forceinline__ void store_order_bytes(uint8_t* p, uint64_t packed)
{
    if constexpr (N == 1) {
        stream_store((uint8_t)packed, p);
    } else if constexpr (N == 2) {
        stream_store((uint16_t)packed, reinterpret_cast<uint16_t*>(p));
    } else if constexpr (N == 4) {
        stream_store((uint32_t)packed, reinterpret_cast<uint32_t*>(p));
    } else if constexpr (N == 8) {
        stream_store(packed, reinterpret_cast<uint64_t*>(p));
    } else {
#pragma unroll
        for (int r = 0; r < N; ++r) p[r] = (uint8_t)(packed >> (8 * r));
    }
}

// The kept indices of a group in selection order (rank r at byte r).
template <int M, int N>
__device__ __forceinline__ void store_idx(uint8_t* p, const int (&rank)[M])
{
    uint64_t packed = 0;
#pragma unroll
    for (int j = 0; j < M; ++j)
        packed |= (rank[j] < N) ? ((uint64_t)j << (8 * rank[j])) : 0ull;
    store_order_bytes<N>(p, packed);
}

// W with the entries outside keep_bits cleared (m = 8).
__device__ __forceinline__ void store_kept8(uint16_t* p, const uint32_t (&w)[8], uint32_t keep_bits)
{
    uint32_t packed[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const uint32_t mask = ((keep_bits >> (2 * t)) & 1u ? 0x0000FFFFu : 0u) |
                              ((keep_bits >> (2 * t + 1)) & 1u ? 0xFFFF0000u : 0u);
        packed[t] = (w[2 * t] | (w[2 * t + 1] << 16)) & mask;
    }
    const u32x4 v = {packed[0], packed[1], packed[2], packed[3]};
    stream_store(v, reinterpret_cast<u32x4*>(p));
}

// The m Philox words of a group (block = its first Philox block index).
template <int M>
__device__ __forceinline__ void group_words(uint32_t block, const NoiseKey& key, uint32_t (&x)[M])
{
#pragma unroll
    for (int t = 0; t < M / 4; ++t) {
        const uint4 v = philox_block(block + t, key);
        x[4 * t + 0] = v.x;
        x[4 * t + 1] = v.y;
        x[4 * t + 2] = v.z;
        x[4 * t + 3] = v.w;
    }
}

// The exact keys kappa = fl(fl(phi / lambda) + g) (noise.hpp).
template <int M, bool kLambdaOne>
__device__ __forceinline__ void exact_keys(const float (&phi)[M], const uint32_t (&x)[M],
                                           float lambda, const float2* tab, float (&kappa)[M])
{
#pragma unroll
    for (int j = 0; j < M; ++j) kappa[j] = key_of<kLambdaOne>(phi[j], lambda, x[j], tab);
}

// The hardware-log keys in log2 units (noise.hpp).
template <int M>
__device__ __forceinline__ void fast_keys(const float (&phi)[M], const uint32_t (&x)[M], float c,
                                          float (&k)[M])
{
#pragma unroll
    for (int j = 0; j < M; ++j) k[j] = fast_key_log2(phi[j], c, x[j]);
}

// Hard top-n of eight hardware-log keys by sorting 32-bit integers: each key's
// bits mapped to an unsigned integer of the same order, the low 3 bits
// replaced by the entry's index, then the 19 comparators of an 8-input sorting
// network (Knuth, TAOCP vol. 3, 5.3.4), each one unsigned max and min.
// Clearing the 3 bits lowers a key by less than 8 ulps (2^-20 |K|), so the
// margin of noise.hpp widens to kFastPairMargin + 2^-19 max|K|, checked on
// the 7 pairs adjacent in sorted order.  Returns whether the keys are that
// far apart (then the order is the exact keys' order and none tie); sets
// keep_bits (bit j: entry j is among the n largest) and order (the indices
// of ranks 0..n-1, one per byte).
__device__ __forceinline__ uint32_t sortable_bits(float f)
{
    const uint32_t u = __float_as_uint(f);
    return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u); // negative: ~u; else set the sign bit
}

__device__ __forceinline__ float float_of_sortable(uint32_t v)
{
    return __uint_as_float(v ^ (~(uint32_t)((int32_t)v >> 31) | 0x80000000u));
}

template <int I, int J>
__device__ __forceinline__ void sort_pair_desc(uint32_t (&p)[8])
{
    const uint32_t a = p[I], b = p[J];
    p[I] = a > b ? a : b;
    p[J] = a > b ? b : a;
}

template <int N>
__device__ __forceinline__ bool top8_fast(const float (&k)[8], uint32_t& keep_bits, uint64_t& order)
{
    uint32_t p[8];
    float big = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        p[j] = (sortable_bits(k[j]) & ~7u) | (uint32_t)j;
        big = fmaxf(big, fabsf(k[j]));
    }
    sort_pair_desc<0, 2>(p); sort_pair_desc<1, 3>(p); sort_pair_desc<4, 6>(p); sort_pair_desc<5, 7>(p);
    sort_pair_desc<0, 4>(p); sort_pair_desc<1, 5>(p); sort_pair_desc<2, 6>(p); sort_pair_desc<3, 7>(p);
    sort_pair_desc<0, 1>(p); sort_pair_desc<2, 3>(p); sort_pair_desc<4, 5>(p); sort_pair_desc<6, 7>(p);
    sort_pair_desc<2, 4>(p); sort_pair_desc<3, 5>(p);
    sort_pair_desc<1, 4>(p); sort_pair_desc<3, 6>(p);
    sort_pair_desc<1, 2>(p); sort_pair_desc<3, 4>(p); sort_pair_desc<5, 6>(p);
    const float margin = __builtin_fmaf(big, 0x1p-19f, kFastPairMargin);
    bool sep = true;
    float prev = float_of_sortable(p[0] & ~7u);
#pragma unroll
    for (int r = 1; r < 8; ++r) {
        const float cur = float_of_sortable(p[r] & ~7u);
        sep &= prev - cur > margin;
        prev = cur;
    }
    keep_bits = 0u;
    order = 0u;
#pragma unroll
    for (int r = 0; r < N; ++r) {
        keep_bits |= 1u << (p[r] & 7u);
        order |= (uint64_t)(p[r] & 7u) << (8 * r);
    }
    return sep;
}

// A block works on one piece of the batch (common.hpp).  Each iteration of a
// block covers U * kLaneBlock consecutive groups of the piece: lane l takes
// groups base + u * kLaneBlock + l, u < U, so every load and store instruction
// of a wave is one contiguous span, and all of a lane's loads are issued
// before its first group is computed (more bytes in flight per wave).
//
// The relaxation takes the exp-domain recursion in groups whose key spans
// allow it, else the log-domain one (relax.hpp); kQ is 1 or 2 for tau = 1 or
// 1/2 (powers by multiplication), else 0.  The choice is made per group, from
// the group's own keys, so a group's outputs never depend on which groups
// share its wave (any split of a tensor into calls gives the same bits).
template <int M, int N, bool kRelax, bool kWantIdx, bool kLambdaOne, int kQ>
__global__ __launch_bounds__(kLaneBlock) void fwd_lane_kernel(FwdBatch a)
{
    // Tables.  With the relaxation every group reads the log cells (exact
    // keys), so the block copies them, and at m = 4 the top-2-of-4 table, into
    // LDS.  Without it the cells serve only groups with near ties and are read
    // from global memory, where they stay cached; and at m = 4 lane e of each
    // wave holds entry e of the 64-entry top-2 table in registers, a group
    // reading entry `code` from lane `code` (ds_bpermute, with every lane of
    // the wave active).  A block then starts streaming without filling LDS or
    // waiting at a barrier.
    constexpr bool kLds = kRelax;
    constexpr bool kLaneTable = M == 4 && !kRelax;
    __shared__ float2 tab_lds[kLds ? kLogCells : 1];
    __shared__ Top4Entry top4[M == 4 && kLds ? 64 : 1];
    const float2* tab = kLds ? tab_lds : kLogCellTable.cell;
    if constexpr (kLds) {
        fill_log_table(tab_lds);
        if constexpr (M == 4) {
            if (threadIdx.x >= kLogCells && threadIdx.x < kLogCells + 64)
                top4[threadIdx.x - kLogCells] = kTop4Table<N>.e[threadIdx.x - kLogCells];
        }
        __syncthreads();
    }
    Top4Entry lane_entry{};
    if constexpr (kLaneTable) lane_entry = kTop4Table<N>.e[threadIdx.x & 63];
    const FwdPiece& pc = a.p[find_piece(a)];
    NoiseKey key = a.key_base;
    key.block_hi = pc.block_hi;
    const int64_t ng = pc.ngroups;
    constexpr int U = kUnrollFwd<M>;
    const int64_t chunk = (int64_t)kLaneBlock * U;
    for (int64_t base = (int64_t)(blockIdx.x - pc.first_block) * chunk; base < ng;
         base += (int64_t)pc.nblocks * chunk) {
        float phi[U][M];
        uint32_t w[U][M];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t q = base + u * kLaneBlock + threadIdx.x;
            if (q < ng) {
                load_logits<M>(pc.phi + q * M, phi[u]);
                load_bf16<M>(pc.W + q * M, w[u]);
            } else if constexpr (kLaneTable) { // a group past the end still looks up
#pragma unroll
                for (int j = 0; j < M; ++j) {
                    phi[u][j] = 0.0f;
                    w[u][j] = 0u;
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t q = base + u * kLaneBlock + threadIdx.x;
            if (!kLaneTable && q >= ng) continue;
            uint32_t x[M];
            group_words<M>(pc.block0 + (uint32_t)q * (M / 4), key, x);
            if constexpr (M == 8 && !kRelax) {
                // Sort the hardware-log keys; a group with a pair closer than
                // the margin takes the exact keys and their ranks instead.
                float kf[8];
                fast_keys<8>(phi[u], x, a.key_c, kf);
                uint32_t keep_bits;
                uint64_t order;
                if (top8_fast<N>(kf, keep_bits, order)) {
                    store_kept8(pc.Wm + q * M, w[u], keep_bits);
                    if (kWantIdx) store_order_bytes<N>(pc.idx + q * N, order);
                } else {
                    float kappa[8];
                    int rank[8];
                    exact_keys<8, kLambdaOne>(phi[u], x, a.lambda, tab, kappa);
                    rank_keys<8>(kappa, rank);
                    store_masked<8>(pc.Wm + q * M, w[u], rank, N);
                    if (kWantIdx) store_idx<8, N>(pc.idx + q * N, rank);
                }
                continue;
            }
            float kappa[M];
            if constexpr (kRelax) {
                // the relaxation's soft mask is an fp32 output: exact keys
                exact_keys<M, kLambdaOne>(phi[u], x, a.lambda, tab, kappa);
            } else {
                // Comparisons only: the hardware keys order every pair that is
                // further apart than their error margin exactly as the exact keys
                // do; a group with a closer pair (rare) takes the exact keys.
                fast_keys<M>(phi[u], x, a.key_c, kappa);
                if (!fast_keys_separated<M>(kappa))
                    exact_keys<M, kLambdaOne>(phi[u], x, a.lambda, tab, kappa);
            }
            const bool soft = kRelax && a.soft;
            if constexpr (kLaneTable) {
                const int addr = (int)(top4_code(kappa) << 2); // byte address of lane `code`
                const uint32_t m01 =
                    (uint32_t)__builtin_amdgcn_ds_bpermute(addr, (int)lane_entry.m01);
                const uint32_t m23 =
                    (uint32_t)__builtin_amdgcn_ds_bpermute(addr, (int)lane_entry.m23);
                const uint32_t order =
                    kWantIdx ? (uint32_t)__builtin_amdgcn_ds_bpermute(addr, (int)lane_entry.order)
                             : 0u;
                if (q < ng) {
                    const u32x2 v = {(w[u][0] | (w[u][1] << 16)) & m01,
                                     (w[u][2] | (w[u][3] << 16)) & m23};
                    stream_store(v, reinterpret_cast<u32x2*>(pc.Wm + q * M));
                    if (kWantIdx) store_order<N>(pc.idx + q * N, order);
                }
            } else if constexpr (M == 4) {
                const Top4Entry t4 = top4[top4_code(kappa)];
                if (!soft) {
                    const u32x2 v = {(w[u][0] | (w[u][1] << 16)) & t4.m01,
                                     (w[u][2] | (w[u][3] << 16)) & t4.m23};
                    stream_store(v, reinterpret_cast<u32x2*>(pc.Wm + q * M));
                }
                if (kWantIdx) store_order<N>(pc.idx + q * N, t4.order);
            } else {
                int rank[M];
                rank_keys<M>(kappa, rank);
                if (!soft) store_masked<M>(pc.Wm + q * M, w[u], rank, N);
                if (kWantIdx) store_idx<M, N>(pc.idx + q * N, rank);
            }
            if (kRelax) {
                float S[M], b[M], bmax;
                StepRec<M> unused[N]; // not written when records are not kept
                const float span = scaled_keys<M>(kappa, a.key_scale, b, bmax);
                if (span <= a.exp_span)
                    relax_forward_exp<M, N, true, false, kQ>(b, bmax, a.inv_tau, S, unused);
                else
                    relax_forward<M, N, true, false>(b, bmax, a.inv_tau, S, unused);
                if (pc.S) {
                    f32x4* s4 = reinterpret_cast<f32x4*>(pc.S + q * M);
#pragma unroll
                    for (int t = 0; t < M / 4; ++t) {
                        const f32x4 v = {S[4 * t], S[4 * t + 1], S[4 * t + 2], S[4 * t + 3]};
                        stream_store(v, s4 + t);
                    }
                }
                if (soft) { // pure soft forward: W (.) S, rounded to bf16
                    uint32_t wp[M / 2];
#pragma unroll
                    for (int i = 0; i < M / 2; ++i) wp[i] = w[u][2 * i] | (w[u][2 * i + 1] << 16);
                    store_soft_product<M>(pc.Wm + q * M, wp, S);
                }
            }
        }
    }
}

// Keys from the logits and the noise ng = -g of m elements (four at a time).
template <int M>
__device__ __forceinline__ void keys_from_noise(const float (&phi)[M], const float (&ng)[M],
                                                float lambda, float (&kappa)[M])
{
#pragma unroll
    for (int t = 0; t < M / 4; ++t) {
        const float p4[4] = {phi[4 * t], phi[4 * t + 1], phi[4 * t + 2], phi[4 * t + 3]};
        float a4[4];
        scaled_logits4(p4, lambda, a4);
#pragma unroll
        for (int e = 0; e < 4; ++e) kappa[4 * t + e] = a4[e] - ng[4 * t + e];
    }
}

// One chunk of the soft forward alone: U groups per lane, loads first (the
// log cells, then the groups' inputs), the noise while they are in flight,
// no per-lane condition in a full chunk (see bwd_lane_span).
template <int M, int N, int kQ, bool kFull>
__device__ __forceinline__ void soft_lane_chunk(const FwdBatch& a, const FwdPiece& pc,
                                                const NoiseKey& key, float2* tab, int64_t base,
                                                int64_t ng_total)
{
    constexpr int U = kUnrollFwd<M>;
    const float4 cells = log_cells_of_lane();
    __builtin_amdgcn_sched_barrier(0);
    float phi[U][M];
    uint32_t w[U][M / 2];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t q = base + u * kLaneBlock + threadIdx.x;
        if (kFull || q < ng_total) {
            load_logits<M>(pc.phi + q * M, phi[u]);
            load_bf16_pairs<M>(pc.W + q * M, w[u]);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    float ng[U][M];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t q = base + u * kLaneBlock + threadIdx.x;
        uint32_t x[M];
        group_words<M>(pc.block0 + (uint32_t)q * (M / 4), key, x);
        if (u == 0) publish_log_table(tab, cells);
#pragma unroll
        for (int j = 0; j < M; ++j) ng[u][j] = neg_gumbel_from_word(x[j], tab);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t q = base + u * kLaneBlock + threadIdx.x;
        if (!kFull && q >= ng_total) continue;
        float kappa[M];
        keys_from_noise<M>(phi[u], ng[u], a.lambda, kappa);
        float S[M], b[M], bmax;
        StepRec<M> unused[N]; // not written when records are not kept
        if constexpr (kQ < 0) {
            scaled_keys<M, false>(kappa, a.key_scale, b, bmax);
            relax_forward<M, N, true, false>(b, bmax, a.inv_tau, S, unused);
        } else if (scaled_keys<M>(kappa, a.key_scale, b, bmax) <= a.exp_span) {
            relax_forward_exp<M, N, true, false, kQ>(b, bmax, a.inv_tau, S, unused);
        } else {
            relax_forward<M, N, true, false>(b, bmax, a.inv_tau, S, unused);
        }
        store_soft_product<M>(pc.Wm + q * M, w[u], S);
    }
}

// Pure soft forward whose only output is W_soft = bf16(W (.) S) (neither S
// nor the indices requested): the relaxation at the exact keys, with no
// selection.  The block's waves share one copy of the log cells in LDS
// (noise.hpp), so a block starts streaming without a barrier.
template <int M, int N, int kQ>
__global__ __launch_bounds__(kLaneBlock) void fwd_soft_lane_kernel(FwdBatch a)
{
    __shared__ float4 tab4[kLogCells / 2];
    float2* tab = reinterpret_cast<float2*>(tab4);
    const FwdPiece& pc = a.p[find_piece(a)];
    NoiseKey key = a.key_base;
    key.block_hi = pc.block_hi;
    const int64_t ng = pc.ngroups;
    const int64_t chunk = (int64_t)kLaneBlock * kUnrollFwd<M>;
    for (int64_t base = (int64_t)(blockIdx.x - pc.first_block) * chunk; base < ng;
         base += (int64_t)pc.nblocks * chunk) {
        if (base + chunk <= ng)
            soft_lane_chunk<M, N, kQ, true>(a, pc, key, tab, base, ng);
        else
            soft_lane_chunk<M, N, kQ, false>(a, pc, key, tab, base, ng);
    }
}

// The backward of one group of 4 (and, with kAdam, its AdamW step), given
// the group's noise: ng = -g, computed before its inputs arrive.  kQ: the
// exp-domain power mode of tau (relax.hpp), or -1 where that form is off.
template <int N, bool kLambdaOne, bool kAdam, int kQ>
__device__ __forceinline__ void bwd_group4(const BwdBatch& a, const BwdPiece& pc,
                                           const float (&ng)[4], const BwdSlot<kAdam>& in,
                                           int64_t q)
{
    constexpr int M = 4;
    float phi[M] = {in.phi.x, in.phi.y, in.phi.z, in.phi.w};
    // the keys the forward sampled: kappa = fl(fl(phi / lambda) + g) (noise.hpp)
    float kappa[M];
#pragma unroll
    for (int j = 0; j < M; ++j) kappa[j] = (kLambdaOne ? phi[j] : phi[j] / a.lambda) - ng[j];
    // Straight-through: dL/dS = dL/dW_masked (.) W, exact in fp32 (bf16 x bf16).
    const uint32_t w[M] = {in.w.x & 0xFFFFu, in.w.x >> 16, in.w.y & 0xFFFFu, in.w.y >> 16};
    const uint32_t g[M] = {in.g.x & 0xFFFFu, in.g.x >> 16, in.g.y & 0xFFFFu, in.g.y >> 16};
    float sbar[M];
#pragma unroll
    for (int j = 0; j < M; ++j) sbar[j] = bf16_bits_to_float(g[j]) * bf16_bits_to_float(w[j]);
    // Relaxation forward keeping its records, then the reverse sweep: the
    // exp-domain recursion where the group's key span allows it (the floor of
    // log(1 - mu) is then out of reach), else the log-domain one with the
    // floor's case in the sweep (relax.hpp).
    StepRec<M> rec[N];
    float S_unused[M], b[M], abar[M], bmax;
    if constexpr (kQ < 0) { // the exp-domain form is off at this temperature
        scaled_keys<M, false>(kappa, a.key_scale, b, bmax);
        relax_forward<M, N, false, true>(b, bmax, a.inv_tau, S_unused, rec);
        relax_backward<M, N, false, true>(rec, sbar, a.inv_tau, abar);
    } else if (scaled_keys<M>(kappa, a.key_scale, b, bmax) <= a.exp_span) {
        relax_forward_exp<M, N, false, true, kQ>(b, bmax, a.inv_tau, S_unused, rec);
        relax_backward<M, N, kQ == 1, false>(rec, sbar, a.inv_tau, abar);
    } else {
        relax_forward<M, N, false, true>(b, bmax, a.inv_tau, S_unused, rec);
        relax_backward<M, N, false, true>(rec, sbar, a.inv_tau, abar);
    }
    float grad[M]; // dL/dphi = dL/dkappa / lambda
#pragma unroll
    for (int j = 0; j < M; ++j) grad[j] = kLambdaOne ? abar[j] : abar[j] * a.inv_lambda;
    if (!kAdam || pc.dphi) store_f32<M>(pc.dphi + q * M, grad);
    if constexpr (kAdam) {
        float mom[M] = {in.mom.x, in.mom.y, in.mom.z, in.mom.w};
        float sec[M] = {in.sec.x, in.sec.y, in.sec.z, in.sec.w};
#pragma unroll
        for (int j = 0; j < M; ++j) adamw_update(a.adam, grad[j], phi[j], mom[j], sec[j]);
        store_f32<M>(const_cast<float*>(pc.phi) + q * M, phi);
        store_f32<M>(pc.m + q * M, mom);
        store_f32<M>(pc.v + q * M, sec);
    }
}

// The noise of a lane's group (ng = -g for its four elements, noise.hpp).
__device__ __forceinline__ void group_noise4(uint32_t block, const NoiseKey& key, const float2* tab,
                                             float (&ng)[4])
{
    uint32_t x[4];
    group_words<4>(block, key, x);
#pragma unroll
    for (int j = 0; j < 4; ++j) ng[j] = neg_gumbel_from_word(x[j], tab);
}

// kBwdChunks chunks of kLaneBlock groups from `base`, one group per lane and
// chunk.  The loads go out first (the group's inputs, the log cells, and with
// more than one chunk the next chunk's inputs); the noise -- the Philox words
// and both logarithms of every element, about half of the arithmetic --
// needs none of them, so each chunk's noise runs while loads are in flight.
// kFull: every group of the span is inside the piece, so there is no
// per-lane condition and each wait for a load is exactly for that load (a
// condition around a load makes the compiler wait for every load at the
// join).
template <int N, bool kLambdaOne, bool kAdam, int kQ, bool kFull>
__device__ __forceinline__ void bwd_lane_span(const BwdBatch& a, const BwdPiece& pc,
                                              const NoiseKey& key, float2* tab, int64_t base,
                                              int64_t ng_total)
{
    constexpr int K = kBwdChunks;
    const int64_t q0 = base + threadIdx.x;
    BwdSlot<kAdam> in[2];
    if (kFull || q0 < ng_total) load_bwd_slot<kAdam>(pc, q0, in[0]);
    __builtin_amdgcn_sched_barrier(0);
    const float4 cells = log_cells_of_lane();
    __builtin_amdgcn_sched_barrier(0);
    if (K > 1 && (kFull || q0 + kLaneBlock < ng_total))
        load_bwd_slot<kAdam>(pc, q0 + kLaneBlock, in[1]);
    __builtin_amdgcn_sched_barrier(0);
    float ng[2][4];
    {
        uint32_t x[4];
        group_words<4>(pc.block0 + (uint32_t)q0, key, x);
        publish_log_table(tab, cells);
#pragma unroll
        for (int j = 0; j < 4; ++j) ng[0][j] = neg_gumbel_from_word(x[j], tab);
    }
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int64_t q = q0 + (int64_t)k * kLaneBlock;
        if (k + 1 < K) group_noise4(pc.block0 + (uint32_t)(q + kLaneBlock), key, tab, ng[(k + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
        if (kFull || q < ng_total)
            bwd_group4<N, kLambdaOne, kAdam, kQ>(a, pc, ng[k & 1], in[k & 1], q);
        if (k + 2 < K && (kFull || q + 2 * kLaneBlock < ng_total))
            load_bwd_slot<kAdam>(pc, q + 2 * kLaneBlock, in[k & 1]);
    }
}

// Backward for m = 4 (m = 8 and wider take the kernels of wide_bwd.hip);
// with kAdam the AdamW step on the logits is fused in: the moments are read
// with the group's other inputs, and the updated logits and moments are
// written instead of (or besides, when pc.dphi is set) the gradient.  kQ as
// in fwd_lane_kernel.  A block takes kBwdChunks consecutive chunks of
// kLaneBlock groups.
template <int M, int N, bool kLambdaOne, bool kAdam, int kQ>
__global__ __launch_bounds__(kLaneBlock) void bwd_lane_kernel(BwdBatch a)
{
    static_assert(M == 4, "the lane backward serves m = 4");
    // Every group takes the exact keys; the block's waves share one copy of
    // the log cells in LDS (noise.hpp).
    __shared__ float4 tab4[kLogCells / 2];
    float2* tab = reinterpret_cast<float2*>(tab4);
    const BwdPiece& pc = a.p[find_piece(a)];
    NoiseKey key = a.key_base;
    key.block_hi = pc.block_hi;
    const int64_t ng = pc.ngroups;
    const int64_t span = (int64_t)kLaneBlock * kBwdChunks;
    for (int64_t base = (int64_t)(blockIdx.x - pc.first_block) * span; base < ng;
         base += (int64_t)pc.nblocks * span) {
        if (base + span <= ng)
            bwd_lane_span<N, kLambdaOne, kAdam, kQ, true>(a, pc, key, tab, base, ng);
        else
            bwd_lane_span<N, kLambdaOne, kAdam, kQ, false>(a, pc, key, tab, base, ng);
    }
}

// Noise inspection: one Philox call per 4 consecutive elements.
__global__ __launch_bounds__(kBlock) void noise_kernel(uint32_t* words, float* gum, int64_t count,
                                                       uint32_t block0, NoiseKey key)
{
    __shared__ float2 tab[kLogCells];
    fill_log_table(tab);
    __syncthreads();
    const int64_t nblocks = (count + 3) / 4;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t b = (int64_t)blockIdx.x * kBlock + threadIdx.x; b < nblocks; b += stride) {
        const uint4 x = philox_block(block0 + (uint32_t)b, key);
        const uint32_t xs[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int64_t e = 4 * b + t;
            if (e < count) {
                if (words) words[e] = xs[t];
                if (gum) gum[e] = gumbel_from_word(xs[t], tab);
            }
        }
    }
}

__global__ __launch_bounds__(kBlock) void fast_noise_kernel(const uint32_t* words, float* out,
                                                            int64_t count)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < count; i += stride)
        out[i] = fast_noise_log2(words[i]);
}

__global__ __launch_bounds__(kBlock) void gumbel_words_kernel(const uint32_t* words, float* gum,
                                                              int64_t count)
{
    __shared__ float2 tab[kLogCells];
    fill_log_table(tab);
    __syncthreads();
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < count; i += stride)
        gum[i] = gumbel_from_word(words[i], tab);
}

// ----------------------------------------------------------------------------- host side
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ---- dispatch tables over (m, n) and the boolean variants

// How the exp-domain recursion raises omega to 1 / tau: 1 or 2 when 1 / tau
// is that integer (by multiplication), else 0 (exp2 and log2).
// -1 where the exp-domain form is off (q = 1 / tau above 2.25, see
// exp_span_limit): the backward and the soft forward alone then have a
// log-domain-only variant.  The other forwards treat -1 as 0 (their
// exp-domain branch is never taken there).
int tau_mode(float tau)
{
    if (tau == 1.0f) return 1;
    if (tau == 0.5f) return 2;
    return 1.0 / (double)tau > 2.25 ? -1 : 0;
}

// Largest key span (units of b, relax.hpp) for which a group may take the
// exp-domain recursion: kExpSpanAccuracy, and kExpNormalBound - log2 m -
// (n - 1) q with q = 1 / tau (without an update step, n = 1, only the first
// applies).  For
// q > 2.25 the bound admits only key spans below 10 (natural units; 32 /
// (q log2 e)), a few times the spread of the keys themselves, so many waves
// would mix groups of both kinds and run both recursions; there the
// exp-domain form is off (-1 admits no group).  The limit depends only on
// (n, tau).
float exp_span_limit(int n, int m, float tau)
{
    const double q = 1.0 / (double)tau;
    if (q > 2.25) return -1.0f;
    const double repr =
        n <= 1 ? INFINITY : (double)kExpNormalBound - std::log2((double)m) - (n - 1) * q;
    return (float)std::min((double)kExpSpanAccuracy, repr);
}

template <int M, int N, bool S, bool I, bool L>
FwdFn pick_fwd_q(int q)
{
    if constexpr (!S) return fwd_lane_kernel<M, N, S, I, L, 0>; // no relaxation
    else
        return q == 1 ? fwd_lane_kernel<M, N, S, I, L, 1>
                      : (q == 2 ? fwd_lane_kernel<M, N, S, I, L, 2> : fwd_lane_kernel<M, N, S, I, L, 0>);
}

template <int M, int N>
FwdFn pick_fwd(bool want_s, bool want_idx, bool lam1, int q)
{
#define ROI_FWD(S, I, L) \
    if (want_s == S && want_idx == I && lam1 == L) return pick_fwd_q<M, N, S, I, L>(q);
    ROI_FWD(false, false, false) ROI_FWD(false, false, true) ROI_FWD(false, true, false)
    ROI_FWD(false, true, true) ROI_FWD(true, false, false) ROI_FWD(true, false, true)
    ROI_FWD(true, true, false) ROI_FWD(true, true, true)
#undef ROI_FWD
    return nullptr;
}

template <int M, int N, bool L, bool A>
BwdFn pick_bwd_q(int q)
{
    if (q < 0) return bwd_lane_kernel<M, N, L, A, -1>;
    return q == 1 ? bwd_lane_kernel<M, N, L, A, 1>
                  : (q == 2 ? bwd_lane_kernel<M, N, L, A, 2> : bwd_lane_kernel<M, N, L, A, 0>);
}

template <int M, int N>
BwdFn pick_bwd(bool lam1, bool adam, int q)
{
    if (adam) return lam1 ? pick_bwd_q<M, N, true, true>(q) : pick_bwd_q<M, N, false, true>(q);
    return lam1 ? pick_bwd_q<M, N, true, false>(q) : pick_bwd_q<M, N, false, false>(q);
}

template <int M, int... Ns>
FwdFn fwd_for_n(int n, bool s, bool i, bool l, int q, std::integer_sequence<int, Ns...>)
{
    FwdFn f = nullptr;
    ((n == Ns + 1 ? (f = pick_fwd<M, Ns + 1>(s, i, l, q), 0) : 0), ...);
    return f;
}

template <int M, int... Ns>
BwdFn bwd_for_n(int n, bool l, bool adam, int q, std::integer_sequence<int, Ns...>)
{
    BwdFn f = nullptr;
    ((n == Ns + 1 ? (f = pick_bwd<M, Ns + 1>(l, adam, q), 0) : 0), ...);
    return f;
}

template <int M, int N>
FwdFn pick_soft(int q)
{
    if (q < 0) return fwd_soft_lane_kernel<M, N, -1>;
    return q == 1 ? fwd_soft_lane_kernel<M, N, 1>
                  : (q == 2 ? fwd_soft_lane_kernel<M, N, 2> : fwd_soft_lane_kernel<M, N, 0>);
}

template <int M, int... Ns>
FwdFn soft_for_n(int n, int q, std::integer_sequence<int, Ns...>)
{
    FwdFn f = nullptr;
    ((n == Ns + 1 ? (f = pick_soft<M, Ns + 1>(q), 0) : 0), ...);
    return f;
}

// The soft forward with no output but W_soft.
FwdFn select_soft_only(int m, int n, float tau)
{
    const int q = tau_mode(tau);
    if (m == 4) return soft_for_n<4>(n, q, std::make_integer_sequence<int, 4>{});
    if (m == 8) return soft_for_n<8>(n, q, std::make_integer_sequence<int, 8>{});
    return select_wide_soft_only(m, n, q);
}

FwdFn select_fwd(int m, int n, bool s, bool i, bool l, float tau)
{
    const int q = std::max(0, tau_mode(tau));
    if (m == 4) return fwd_for_n<4>(n, s, i, l, q, std::make_integer_sequence<int, 4>{});
    if (m == 8) return fwd_for_n<8>(n, s, i, l, q, std::make_integer_sequence<int, 8>{});
    return select_wide_fwd(m, n, s, q);
}

BwdFn select_bwd(int m, int n, bool l, bool adam, float tau)
{
    const int q = tau_mode(tau);
    if (m == 4) return bwd_for_n<4>(n, l, adam, q, std::make_integer_sequence<int, 4>{});
    return select_wide_bwd(m, n, adam, q);
}

} // namespace
} // namespace roi

using namespace roi;

namespace roi {
namespace {

// Blocks one piece of `ngroups` groups needs in a launch.
int64_t blocks_for(int64_t ngroups, int m, bool fwd)
{
    if (m > 8 || (m == 8 && !fwd)) // wide kernels: m / 4 slots per group
        return ceil_div(ngroups * (m / 4), fwd ? (int64_t)kBlock : wide_bwd_block_slots(m));
    const int u = fwd ? (m == 4 ? kUnrollFwd<4> : kUnrollFwd<8>) : kBwdChunks;
    return ceil_div(ngroups, (int64_t)u * kLaneBlock);
}

// Collects pieces into batches of up to kMaxPieces and launches each batch as
// one grid (kept below 2^32 threads; a piece that alone needs more blocks
// gets the largest grid and its blocks stride over it).
template <typename Batch, typename Piece, typename Fn>
struct Launcher {
    Batch batch;
    Fn fn;
    int block;
    int m;
    bool fwd;
    hipStream_t stream;
    const char* what;
    int64_t blocks = 0;

    int64_t max_blocks() const { return (int64_t)(0xFFFFFFFFu / (uint32_t)block); }

    int flush()
    {
        if (batch.count == 0) return ROI_OK;
        void* args[] = {&batch};
        const hipError_t e = hipLaunchKernel((const void*)fn, dim3((unsigned)blocks),
                                             dim3(block), args, 0, stream);
        batch.count = 0;
        blocks = 0;
        if (e != hipSuccess) return launch_status(what);
        return launch_status(what);
    }

    int add(Piece pc)
    {
        const int64_t nb = std::min(blocks_for(pc.ngroups, m, fwd), max_blocks());
        if (batch.count == kMaxPieces || blocks + nb > max_blocks())
            if (int st = flush()) return st;
        if (batch.count == 0)
            for (uint32_t& s : batch.starts) s = 0xFFFFFFFFu;
        pc.first_block = (uint32_t)blocks;
        pc.nblocks = (uint32_t)nb;
        batch.starts[batch.count] = pc.first_block;
        batch.p[batch.count++] = pc;
        blocks += nb;
        return ROI_OK;
    }
};

int mask_fwd_run(const char* what, bool soft, const roi_fwd_tensor* t, int count, int n, int m,
                 float tau, float lambda, uint64_t seed, uint64_t step, hipStream_t stream)
{
    int with_s, with_idx;
    if (int st = validate_fwd(t, count, n, m, tau, lambda, &with_s, &with_idx)) return st;
    if (with_s < 0) return ok(); // nothing to do
    // The soft forward alone needs no selection: a kernel of its own.
    const bool soft_only = soft && with_s == 0 && with_idx == 0;
    FwdFn fn = soft_only
                   ? select_soft_only(m, n, tau)
                   : select_fwd(m, n, soft || with_s == 1, with_idx == 1, lambda == 1.0f, tau);
    if (!fn) return fail(ROI_E_UNSUPPORTED, "no kernel for %d:%d", n, m);
    Launcher<FwdBatch, FwdPiece, FwdFn> L{};
    L.fn = fn;
    L.block = m > 8 ? kBlock : kLaneBlock;
    L.m = m;
    L.fwd = true;
    L.stream = stream;
    L.what = what;
    L.batch.key_base = make_key(seed, step, 0);
    L.batch.lambda = lambda;
    L.batch.key_c = (float)(1.4426950408889634 / (double)lambda); // log2(e) / lambda
    L.batch.inv_tau = (float)(1.0 / (double)tau);
    L.batch.key_scale = kLog2e * L.batch.inv_tau;
    L.batch.exp_span = exp_span_limit(n, m, tau);
    L.batch.soft = soft ? 1 : 0;
    for (int i = 0; i < count; ++i) {
        const int64_t ngroups = t[i].rows * t[i].cols / m;
        if (ngroups == 0) continue;
        const int st = for_each_piece(t[i].elem_offset, ngroups, m,
                                      [&](int64_t g0, int64_t ng, uint64_t e0) {
            FwdPiece pc{};
            pc.W = t[i].W + g0 * m;
            pc.phi = t[i].logits + g0 * m;
            pc.Wm = t[i].W_masked + g0 * m;
            pc.S = t[i].soft_mask ? t[i].soft_mask + g0 * m : nullptr;
            pc.idx = t[i].sel_idx ? t[i].sel_idx + g0 * n : nullptr;
            pc.ngroups = ng;
            pc.block0 = (uint32_t)(e0 / 4);
            pc.block_hi = (uint32_t)((e0 / 4) >> 32);
            return L.add(pc);
        });
        if (st) return st;
    }
    return L.flush();
}

int mask_bwd_core(const char* what, const BwdDesc* t, int count, int n, int m, float tau,
                  float lambda, uint64_t seed, uint64_t step, const roi_adamw_params* opt,
                  hipStream_t stream)
{
    const bool adam = opt != nullptr;
    AdamStep astep{};
    bool any;
    if (int st = validate_bwd(t, count, n, m, tau, lambda, opt, &astep, &any)) return st;
    if (!any) return ok();
    BwdFn fn = select_bwd(m, n, lambda == 1.0f, adam, tau);
    if (!fn) return fail(ROI_E_UNSUPPORTED, "no kernel for %d:%d", n, m);
    Launcher<BwdBatch, BwdPiece, BwdFn> L{};
    L.fn = fn;
    L.block = m >= 8 ? kBlock : kLaneBlock;
    L.m = m;
    L.fwd = false;
    L.stream = stream;
    L.what = what;
    L.batch.key_base = make_key(seed, step, 0);
    L.batch.lambda = lambda;
    L.batch.inv_lambda = (float)(1.0 / (double)lambda);
    L.batch.tau = tau;
    L.batch.inv_tau = (float)(1.0 / (double)tau);
    L.batch.key_scale = kLog2e * L.batch.inv_tau;
    L.batch.exp_span = exp_span_limit(n, m, tau);
    L.batch.adam = astep;
    for (int i = 0; i < count; ++i) {
        const int64_t ngroups = t[i].rows * t[i].cols / m;
        if (ngroups == 0) continue;
        const int st = for_each_piece(t[i].off, ngroups, m,
                                      [&](int64_t g0, int64_t ng, uint64_t e0) {
            BwdPiece pc{};
            pc.G = t[i].G + g0 * m;
            pc.W = t[i].W + g0 * m;
            pc.phi = t[i].phi + g0 * m;
            pc.dphi = t[i].dphi ? t[i].dphi + g0 * m : nullptr;
            pc.m = adam ? t[i].m + g0 * m : nullptr;
            pc.v = adam ? t[i].v + g0 * m : nullptr;
            pc.ngroups = ng;
            pc.block0 = (uint32_t)(e0 / 4);
            pc.block_hi = (uint32_t)((e0 / 4) >> 32);
            return L.add(pc);
        });
        if (st) return st;
    }
    return L.flush();
}

} // namespace
} // namespace roi

extern "C" int roi_mask_fwd(const uint16_t* W, const float* logits, int64_t rows, int64_t cols,
                            int n, int m, float tau, float lambda, uint64_t seed, uint64_t step,
                            uint64_t elem_offset, uint16_t* W_masked, float* soft_mask,
                            uint8_t* sel_idx, hipStream_t stream)
{
    const roi_fwd_tensor t = {W, logits, W_masked, soft_mask, sel_idx, rows, cols, elem_offset};
    return mask_fwd_run("roi_mask_fwd", false, &t, 1, n, m, tau, lambda, seed, step, stream);
}

extern "C" int roi_mask_fwd_soft(const uint16_t* W, const float* logits, int64_t rows,
                                 int64_t cols, int n, int m, float tau, float lambda,
                                 uint64_t seed, uint64_t step, uint64_t elem_offset,
                                 uint16_t* W_soft, float* soft_mask, uint8_t* sel_idx,
                                 hipStream_t stream)
{
    const roi_fwd_tensor t = {W, logits, W_soft, soft_mask, sel_idx, rows, cols, elem_offset};
    return mask_fwd_run("roi_mask_fwd_soft", true, &t, 1, n, m, tau, lambda, seed, step, stream);
}

extern "C" int roi_mask_fwd_grouped(const roi_fwd_tensor* tensors, int count, int n, int m,
                                    float tau, float lambda, uint64_t seed, uint64_t step,
                                    hipStream_t stream)
{
    return mask_fwd_run("roi_mask_fwd_grouped", false, tensors, count, n, m, tau, lambda, seed,
                        step, stream);
}

extern "C" int roi_mask_fwd_soft_grouped(const roi_fwd_tensor* tensors, int count, int n, int m,
                                         float tau, float lambda, uint64_t seed, uint64_t step,
                                         hipStream_t stream)
{
    return mask_fwd_run("roi_mask_fwd_soft_grouped", true, tensors, count, n, m, tau, lambda,
                        seed, step, stream);
}

extern "C" int roi_mask_bwd(const uint16_t* grad_W_masked, const uint16_t* W, const float* logits,
                            int64_t rows, int64_t cols, int n, int m, float tau, float lambda,
                            uint64_t seed, uint64_t step, uint64_t elem_offset, float* grad_logits,
                            hipStream_t stream)
{
    const BwdDesc t = {grad_W_masked, W, logits, grad_logits, nullptr, nullptr,
                       rows, cols, elem_offset};
    return mask_bwd_core("roi_mask_bwd", &t, 1, n, m, tau, lambda, seed, step, nullptr, stream);
}

extern "C" int roi_mask_bwd_grouped(const roi_bwd_tensor* tensors, int count, int n, int m,
                                    float tau, float lambda, uint64_t seed, uint64_t step,
                                    hipStream_t stream)
{
    if (int st = check_count(tensors, count)) return st;
    std::vector<BwdDesc> d((size_t)count);
    for (int i = 0; i < count; ++i)
        d[i] = {tensors[i].grad_W_masked, tensors[i].W, tensors[i].logits,
                tensors[i].grad_logits, nullptr, nullptr, tensors[i].rows, tensors[i].cols,
                tensors[i].elem_offset};
    return mask_bwd_core("roi_mask_bwd_grouped", d.data(), count, n, m, tau, lambda, seed, step,
                         nullptr, stream);
}

extern "C" int roi_mask_bwd_adamw(const uint16_t* grad_W_masked, const uint16_t* W,
                                  float* logits, float* exp_avg, float* exp_avg_sq,
                                  float* grad_logits, int64_t rows, int64_t cols, int n, int m,
                                  float tau, float lambda, uint64_t seed, uint64_t step,
                                  uint64_t elem_offset, const roi_adamw_params* opt,
                                  hipStream_t stream)
{
    const BwdDesc t = {grad_W_masked, W, logits, grad_logits, exp_avg, exp_avg_sq,
                       rows, cols, elem_offset};
    if (!opt) return fail(ROI_E_INVAL, "the AdamW parameters must not be NULL");
    return mask_bwd_core("roi_mask_bwd_adamw", &t, 1, n, m, tau, lambda, seed, step, opt,
                         stream);
}

extern "C" int roi_mask_bwd_adamw_grouped(const roi_adamw_tensor* tensors, int count, int n,
                                          int m, float tau, float lambda, uint64_t seed,
                                          uint64_t step, const roi_adamw_params* opt,
                                          hipStream_t stream)
{
    if (int st = check_count(tensors, count)) return st;
    if (!opt) return fail(ROI_E_INVAL, "the AdamW parameters must not be NULL");
    std::vector<BwdDesc> d((size_t)count);
    for (int i = 0; i < count; ++i)
        d[i] = {tensors[i].grad_W_masked, tensors[i].W, tensors[i].logits,
                tensors[i].grad_logits, tensors[i].exp_avg, tensors[i].exp_avg_sq,
                tensors[i].rows, tensors[i].cols, tensors[i].elem_offset};
    return mask_bwd_core("roi_mask_bwd_adamw_grouped", d.data(), count, n, m, tau, lambda, seed,
                         step, opt, stream);
}

extern "C" int roi_mask_export(const float* logits, const uint16_t* W, int64_t rows,
                               int64_t cols, int n, int m, uint16_t* W_masked, uint16_t* values,
                               uint8_t* idx, uint32_t* meta, hipStream_t stream)
{
    Shape sh;
    if (int st = check_shape(rows, cols, n, m, 1.0f, 1.0f, 0, &sh)) return st;
    if (meta && !(n == 2 && m == 4))
        return fail(ROI_E_INVAL, "meta is defined for 2:4 only (got %d:%d)", n, m);
    if (!W_masked && !values && !idx && !meta)
        return fail(ROI_E_INVAL, "no output requested");
    if (sh.numel == 0) return ok();
    if (!logits || (!W && (W_masked || values)))
        return fail(ROI_E_INVAL, "logits (and W, for weight outputs) must not be NULL");
    if (!aligned16(logits) || (W && !aligned16(W)) || (W_masked && !aligned16(W_masked)) ||
        (values && !aligned16(values)) || (idx && !aligned16(idx)) || (meta && !aligned16(meta)))
        return fail(ROI_E_INVAL, "device pointers must be 16-byte aligned");
    const size_t nb2 = (size_t)sh.numel * 2, nb4 = (size_t)sh.numel * 4;
    const size_t nkept = (size_t)sh.ngroups * (size_t)n;
    std::vector<Range> ranges;
    add_range(ranges, logits, nb4, false);
    add_range(ranges, W, nb2, false);
    add_range(ranges, W_masked, nb2, true);
    add_range(ranges, values, nkept * 2, true);
    add_range(ranges, idx, nkept, true);
    add_range(ranges, meta, (size_t)((sh.ngroups + 7) / 8) * 4, true);
    if (int st = check_overlaps(ranges)) return st;
    ExportFn fn = select_export(m, n);
    if (!fn) return fail(ROI_E_UNSUPPORTED, "no kernel for %d:%d", n, m);
    ExportArgs a{logits, W, W_masked, values, idx, meta, sh.ngroups};
    void* args[] = {&a};
    if (hipLaunchKernel((const void*)fn, dim3(grid_for(sh.ngroups)), dim3(kBlock), args, 0,
                        stream) != hipSuccess)
        return launch_status("roi_mask_export");
    return launch_status("roi_mask_export");
}

extern "C" int roi_gumbel_noise(uint64_t seed, uint64_t step, uint64_t elem_offset, int64_t count,
                                uint32_t* words, float* gumbel, hipStream_t stream)
{
    if (count < 0) return fail(ROI_E_INVAL, "count must be >= 0");
    if (elem_offset % 4 != 0) return fail(ROI_E_INVAL, "elem_offset must be a multiple of 4");
    if (count > 0 && elem_offset > UINT64_MAX - (uint64_t)count)
        return fail(ROI_E_INVAL, "elem_offset + count overflows 64 bits");
    if (count == 0) return ok();
    if (!words && !gumbel) return fail(ROI_E_INVAL, "words and gumbel are both NULL");
    if ((words && !aligned16(words)) || (gumbel && !aligned16(gumbel)))
        return fail(ROI_E_INVAL, "device pointers must be 16-byte aligned");
    if (overlap(words, (size_t)count * 4, gumbel, (size_t)count * 4))
        return fail(ROI_E_INVAL, "words and gumbel must not overlap");
    return for_each_piece(elem_offset, count, 1, [&](int64_t i0, int64_t cnt, uint64_t e0) {
        hipLaunchKernelGGL(noise_kernel, dim3(grid_for((cnt + 3) / 4)), dim3(kBlock), 0, stream,
                           words ? words + i0 : nullptr, gumbel ? gumbel + i0 : nullptr, cnt,
                           (uint32_t)(e0 / 4), make_key(seed, step, e0 / 4));
        return launch_status("roi_gumbel_noise");
    });
}

extern "C" int roi_gumbel_from_words(const uint32_t* words, int64_t count, float* gumbel,
                                     hipStream_t stream)
{
    if (count < 0) return fail(ROI_E_INVAL, "count must be >= 0");
    if (count == 0) return ok();
    if (!words || !gumbel) return fail(ROI_E_INVAL, "words and gumbel must not be NULL");
    if (!aligned16(words) || !aligned16(gumbel))
        return fail(ROI_E_INVAL, "device pointers must be 16-byte aligned");
    if (overlap(words, (size_t)count * 4, gumbel, (size_t)count * 4))
        return fail(ROI_E_INVAL, "words and gumbel must not overlap");
    hipLaunchKernelGGL(gumbel_words_kernel, dim3(grid_for(count)), dim3(kBlock), 0, stream, words,
                       gumbel, count);
    return launch_status("roi_gumbel_from_words");
}

extern "C" int roi_fast_noise_from_words(const uint32_t* words, int64_t count, float* out,
                                         hipStream_t stream)
{
    if (count < 0) return fail(ROI_E_INVAL, "count must be >= 0");
    if (count == 0) return ok();
    if (!words || !out) return fail(ROI_E_INVAL, "words and out must not be NULL");
    if (!aligned16(words) || !aligned16(out))
        return fail(ROI_E_INVAL, "device pointers must be 16-byte aligned");
    if (overlap(words, (size_t)count * 4, out, (size_t)count * 4))
        return fail(ROI_E_INVAL, "words and out must not overlap");
    hipLaunchKernelGGL(fast_noise_kernel, dim3(grid_for(count)), dim3(kBlock), 0, stream, words,
                       out, count);
    return launch_status("roi_fast_noise_from_words");
}

extern "C" float roi_anneal(float v_init, float v_end, int64_t t, int64_t t_anneal)
{
    if (!(v_init > 0.0f) || !(v_end > 0.0f) || t < 0 || t_anneal <= 0 || !std::isfinite(v_init) ||
        !std::isfinite(v_end))
        return NAN;
    const double vi = v_init, ve = v_end;
    const double v = vi * std::pow(ve / vi, (double)t / (double)t_anneal);
    return (float)(v > ve ? v : ve);
}

extern "C" const char* roi_status_string(int status)
{
    switch (status) {
    case ROI_OK: return "ok";
    case ROI_E_INVAL: return "invalid argument";
    case ROI_E_UNSUPPORTED: return "unsupported pattern";
    case ROI_E_HIP: return "HIP runtime error";
    default: return "unknown status";
    }
}

extern "C" const char* roi_last_error(void) { return g_last_error.c_str(); }

extern "C" int roi_abi_version(void) { return 1; }
