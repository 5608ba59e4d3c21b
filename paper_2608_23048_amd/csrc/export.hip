// export.hip -- gfx950 kernel of the final-mask export.
//
// After training, the sampling temperature lambda has been annealed towards
// 0 (§4.2.3); the sampler's lambda -> 0 limit keeps the n largest logits of
// each group (ties to the lower index, as in the sampler).  This kernel writes
// that mask in the forms a deployment needs: the dense masked weights, the
// compressed weights (the kept values of each group in increasing index
// order) with their indices, and for 2:4 the indices as 2-bit fields, the
// metadata a sparse-matrix core consumes next to the compressed values.
//
// One lane per group (m <= 32 logits in registers), no noise.  The 2:4
// metadata word of 8 consecutive groups is assembled across 8 adjacent lanes.
#include <hip/hip_runtime.h>

#include <utility>

#include "common.hpp"
#include "relax.hpp"
#include "roi.h"

namespace roi {

namespace {

// m bf16 values of a group (16-bit patterns in the low half of each word).
template <int M>
__device__ __forceinline__ void load_group_bf16(const uint16_t* p, uint32_t (&w)[M])
{
    if constexpr (M == 4) {
        const u32x2 v = stream_load(reinterpret_cast<const u32x2*>(p));
        w[0] = v.x & 0xFFFFu; w[1] = v.x >> 16; w[2] = v.y & 0xFFFFu; w[3] = v.y >> 16;
    } else {
#pragma unroll
        for (int t = 0; t < M / 8; ++t) {
            const u32x4 v = stream_load(reinterpret_cast<const u32x4*>(p) + t);
            w[8 * t + 0] = v.x & 0xFFFFu; w[8 * t + 1] = v.x >> 16;
            w[8 * t + 2] = v.y & 0xFFFFu; w[8 * t + 3] = v.y >> 16;
            w[8 * t + 4] = v.z & 0xFFFFu; w[8 * t + 5] = v.z >> 16;
            w[8 * t + 6] = v.w & 0xFFFFu; w[8 * t + 7] = v.w >> 16;
        }
    }
}

template <int M>
__device__ __forceinline__ void store_group_bf16(uint16_t* p, const uint32_t (&w)[M])
{
    if constexpr (M == 4) {
        const u32x2 v = {w[0] | (w[1] << 16), w[2] | (w[3] << 16)};
        stream_store(v, reinterpret_cast<u32x2*>(p));
    } else {
#pragma unroll
        for (int t = 0; t < M / 8; ++t) {
            const u32x4 v = {w[8 * t] | (w[8 * t + 1] << 16), w[8 * t + 2] | (w[8 * t + 3] << 16),
                             w[8 * t + 4] | (w[8 * t + 5] << 16),
                             w[8 * t + 6] | (w[8 * t + 7] << 16)};
            stream_store(v, reinterpret_cast<u32x4*>(p) + t);
        }
    }
}

template <int M, int N>
__global__ __launch_bounds__(kBlock) void export_kernel(ExportArgs a)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    // The loop bound is uniform over the block, so every lane of a wave takes
    // part in the cross-lane metadata assembly, live or not.
    for (int64_t base = (int64_t)blockIdx.x * kBlock; base < a.ngroups; base += stride) {
        const int64_t q = base + threadIdx.x;
        const bool live = q < a.ngroups;
        uint32_t nib = 0;
        if (live) {
            float phi[M];
            uint32_t w[M];
            load_logits<M>(a.phi + q * M, phi);
            // W is read only when a weight output is requested (it may be NULL
            // otherwise)
            if (a.Wm || a.vals) {
                load_group_bf16<M>(a.W + q * M, w);
            } else {
#pragma unroll
                for (int j = 0; j < M; ++j) w[j] = 0;
            }
            int rank[M];
            rank_keys<M>(phi, rank);
            if (a.Wm) {
                uint32_t wm[M];
#pragma unroll
                for (int j = 0; j < M; ++j) wm[j] = rank[j] < N ? w[j] : 0u;
                store_group_bf16<M>(a.Wm + q * M, wm);
            }
            if constexpr (M <= 8) {
                // kept entries in increasing index order, in registers
                uint32_t kv[N], ki[N];
#pragma unroll
                for (int p = 0; p < N; ++p) kv[p] = ki[p] = 0;
                int pos = 0;
#pragma unroll
                for (int j = 0; j < M; ++j) {
                    const bool keep = rank[j] < N;
#pragma unroll
                    for (int p = 0; p < N; ++p) {
                        kv[p] = (keep && pos == p) ? w[j] : kv[p];
                        ki[p] = (keep && pos == p) ? (uint32_t)j : ki[p];
                    }
                    pos += keep ? 1 : 0;
                }
                if (a.vals) {
                    if constexpr (N % 2 == 0) {
#pragma unroll
                        for (int p = 0; p < N; p += 2)
                            stream_store(kv[p] | (kv[p + 1] << 16),
                                         reinterpret_cast<uint32_t*>(a.vals + q * N + p));
                    } else {
#pragma unroll
                        for (int p = 0; p < N; ++p) a.vals[q * N + p] = (uint16_t)kv[p];
                    }
                }
                if (a.idx) {
#pragma unroll
                    for (int p = 0; p < N; ++p) a.idx[q * N + p] = (uint8_t)ki[p];
                }
                if constexpr (M == 4 && N == 2) nib = ki[0] | (ki[1] << 2);
            } else {
                // m = 16, 32: each kept entry goes straight to its compressed slot
                int pos = 0;
#pragma unroll
                for (int j = 0; j < M; ++j) {
                    if (rank[j] < N) {
                        if (a.vals) a.vals[q * N + pos] = (uint16_t)w[j];
                        if (a.idx) a.idx[q * N + pos] = (uint8_t)j;
                        ++pos;
                    }
                }
            }
        }
        if constexpr (M == 4 && N == 2) {
            if (a.meta) { // uniform: the same for every lane
                uint32_t word = nib << (4 * (threadIdx.x & 7));
                word |= (uint32_t)__shfl_xor((int)word, 1);
                word |= (uint32_t)__shfl_xor((int)word, 2);
                word |= (uint32_t)__shfl_xor((int)word, 4);
                if (live && (threadIdx.x & 7) == 0) stream_store(word, a.meta + q / 8);
            }
        }
    }
}

template <int M, int... Ns>
ExportFn export_for_n(int n, std::integer_sequence<int, Ns...>)
{
    ExportFn f = nullptr;
    ((n == Ns + 1 ? (f = export_kernel<M, Ns + 1>, 0) : 0), ...);
    return f;
}

} // namespace

ExportFn select_export(int m, int n)
{
    if (m == 4) return export_for_n<4>(n, std::make_integer_sequence<int, 4>{});
    if (m == 8) return export_for_n<8>(n, std::make_integer_sequence<int, 8>{});
    if (m == 16) return export_for_n<16>(n, std::make_integer_sequence<int, 16>{});
    if (m == 32) return export_for_n<32>(n, std::make_integer_sequence<int, 32>{});
    return nullptr;
}

} // namespace roi
