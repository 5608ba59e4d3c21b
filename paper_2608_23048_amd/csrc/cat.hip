// cat.hip -- gfx950 kernels of the categorical mask sampler, the
// parameterization the paper compares with (appendix, "Optimization
// Efficiency"): one logit alpha_c per feasible n-hot mask c of a group,
// Pr(c) = softmax(alpha)_c, sampled with Gumbel-Softmax.
//
// One lane per group of m in {4, 8} weights; the C = binom(m, n) candidate
// masks are compile-time bitmasks in lexicographic order of their index sets.
// Keys kappa_c = alpha_c / lambda + g_c with the noise of element 4 B Q + c
// (B = ceil(C / 4) Philox blocks per group Q).  The hard sample is the
// candidate of largest key (ties to the lower candidate), the relaxed mask
// S_j = sum_c y_c [j in c] with y = softmax(kappa / tau), and the backward is
// the straight-through derivative through that softmax.  As in the item
// sampler: the forward without S decides with the hardware-log keys when the
// top two are further apart than their error margin (else with the exact
// keys); S and the backward use the exact keys.
#include <hip/hip_runtime.h>

#include <cmath>
#include <utility>

#include "common.hpp"
#include "host.hpp"
#include "noise.hpp"
#include "relax.hpp"
#include "roi.h"

namespace roi {
namespace {

constexpr int binom(int m, int n)
{
    int r = 1;
    for (int k = 1; k <= n; ++k) r = r * (m - n + k) / k;
    return r;
}

template <int M, int N>
struct Candidates {
    static constexpr int C = binom(M, N);
    uint8_t mask[C];
};

// The n-subsets of {0..m-1} in lexicographic order, as bitmasks.
template <int M, int N>
constexpr Candidates<M, N> make_candidates()
{
    Candidates<M, N> t{};
    int idx[8] = {0, 1, 2, 3, 4, 5, 6, 7};
    for (int c = 0; c < Candidates<M, N>::C; ++c) {
        int mask = 0;
        for (int k = 0; k < N; ++k) mask |= 1 << idx[k];
        t.mask[c] = (uint8_t)mask;
        int k = N - 1;
        while (k >= 0 && idx[k] == M - N + k) --k;
        if (k < 0) break;
        ++idx[k];
        for (int r = k + 1; r < N; ++r) idx[r] = idx[r - 1] + 1;
    }
    return t;
}

template <int M, int N>
constexpr Candidates<M, N> kCand = make_candidates<M, N>();

// Philox words for a 64-bit block index (the block of a candidate need not
// share its high word with the rest of the launch).
__device__ __forceinline__ uint4 philox_block64(uint64_t blk, const NoiseKey& key)
{
    return philox4x32_10((uint32_t)blk, (uint32_t)(blk >> 32), key.step_lo, key.step_hi, key.k0,
                         key.k1);
}

// The C logits of a group (fp32, contiguous, 4C bytes from a 4C-byte stride).
template <int C>
__device__ __forceinline__ void load_cat_logits(const float* p, float (&a)[C])
{
    if constexpr (C % 4 == 0) {
#pragma unroll
        for (int t = 0; t < C / 4; ++t) {
            const f32x4 v = stream_load(reinterpret_cast<const f32x4*>(p) + t);
            a[4 * t] = v.x; a[4 * t + 1] = v.y; a[4 * t + 2] = v.z; a[4 * t + 3] = v.w;
        }
    } else if constexpr (C % 2 == 0) {
        typedef float f32x2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int t = 0; t < C / 2; ++t) {
            const f32x2 v = stream_load(reinterpret_cast<const f32x2*>(p) + t);
            a[2 * t] = v.x; a[2 * t + 1] = v.y;
        }
    } else {
#pragma unroll
        for (int c = 0; c < C; ++c) a[c] = stream_load(p + c);
    }
}

template <int C>
__device__ __forceinline__ void store_cat(float* p, const float (&a)[C])
{
    if constexpr (C % 4 == 0) {
#pragma unroll
        for (int t = 0; t < C / 4; ++t) {
            const f32x4 v = {a[4 * t], a[4 * t + 1], a[4 * t + 2], a[4 * t + 3]};
            stream_store(v, reinterpret_cast<f32x4*>(p) + t);
        }
    } else if constexpr (C % 2 == 0) {
        typedef float f32x2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int t = 0; t < C / 2; ++t) {
            const f32x2 v = {a[2 * t], a[2 * t + 1]};
            stream_store(v, reinterpret_cast<f32x2*>(p) + t);
        }
    } else {
#pragma unroll
        for (int c = 0; c < C; ++c) stream_store(a[c], p + c);
    }
}

// Threads per block: the tile of a block's logits (block * C floats) is staged
// through LDS and must fit in 64 KB.
constexpr int cat_block(int C) { return C > 64 ? 128 : 256; }
// Groups with at least 8 logits (32 bytes) are staged: read per lane from
// global memory, their 32-280-byte strides would touch up to 8x more cache
// lines per load instruction than a contiguous 16-byte-per-lane stream.
constexpr bool cat_staged(int C) { return C >= 8; }
// The backward stages 6 candidates (2:4) as well: per lane, its 24-byte
// strides leave every gradient store instruction covering only part of its
// cache lines.  Measured in one session, the backward was 11% faster staged
// and 6-7% faster with only its stores staged; the forward, which reads
// those strides and stores nothing of them, was 23% slower staged.
constexpr bool cat_staged_bwd(int C) { return C >= 6 && C % 2 == 0; }

// Coalesced copies between global memory and a block's LDS tile, in 8-byte
// chunks (every staged C is even, so a group's logits start 8-byte aligned).
typedef float f32x2v __attribute__((ext_vector_type(2)));

template <int B>
__device__ __forceinline__ void tile_in(const float* g, float* lds, int count)
{
    const f32x2v* src = reinterpret_cast<const f32x2v*>(g);
    f32x2v* dst = reinterpret_cast<f32x2v*>(lds);
    for (int i = threadIdx.x; i < count / 2; i += B) dst[i] = stream_load(src + i);
}

template <int B>
__device__ __forceinline__ void tile_out(const float* lds, float* g, int count)
{
    const f32x2v* src = reinterpret_cast<const f32x2v*>(lds);
    f32x2v* dst = reinterpret_cast<f32x2v*>(g);
    for (int i = threadIdx.x; i < count / 2; i += B) stream_store(src[i], dst + i);
}

struct CatArgs {
    const uint16_t* W;
    const float* alpha;
    const uint16_t* G; // backward
    uint16_t* Wm;      // forward
    float* S;
    uint8_t* choice;
    float* dalpha;     // backward
    int64_t ngroups;
    uint64_t group0;   // global index of group 0
    NoiseKey key;      // block_hi unused
    float lambda;
    float key_c;       // fl(log2(e) / lambda)
    float inv_lambda;
    float inv_tau;
};

// The exact keys of one group (the words x come from its B Philox blocks).
template <int C>
__device__ __forceinline__ void cat_exact_keys(const float (&alpha)[C], const uint32_t (&x)[C],
                                               float lambda, const float2* tab, float (&k)[C])
{
    // a wave-uniform branch, so that lambda = 1 does not run the division
    if (__builtin_amdgcn_readfirstlane(__float_as_uint(lambda)) == 0x3F800000u) {
#pragma unroll
        for (int c = 0; c < C; ++c) k[c] = alpha[c] - neg_gumbel_from_word(x[c], tab);
    } else {
#pragma unroll
        for (int c = 0; c < C; ++c) k[c] = alpha[c] / lambda - neg_gumbel_from_word(x[c], tab);
    }
}

template <int C>
__device__ __forceinline__ void cat_words(uint64_t Q, const NoiseKey& key, uint32_t (&x)[C])
{
    constexpr int B = (C + 3) / 4;
#pragma unroll
    for (int b = 0; b < B; ++b) {
        const uint4 v = philox_block64(Q * B + b, key);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int t = 0; t < 4; ++t)
            if (4 * b + t < C) x[4 * b + t] = w[t];
    }
}

// y = softmax(kappa * scale) in place (scale turns key differences into log2
// units over tau).
template <int C>
__device__ __forceinline__ void cat_softmax(float (&k)[C], float scale)
{
    float mx = k[0];
#pragma unroll
    for (int c = 1; c < C; ++c) mx = fmaxf(mx, k[c]);
    float t = 0.0f;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        k[c] = __builtin_amdgcn_exp2f((k[c] - mx) * scale);
        t += k[c];
    }
    const float r = __builtin_amdgcn_rcpf(t);
#pragma unroll
    for (int c = 0; c < C; ++c) k[c] *= r;
}

template <int M, int N, bool kSoft>
__global__ __launch_bounds__(cat_block(Candidates<M, N>::C)) void cat_fwd_kernel(CatArgs a)
{
    constexpr int C = Candidates<M, N>::C;
    constexpr int B = cat_block(C);
    constexpr bool kStage = cat_staged(C);
    // The log cells in LDS only when every group takes the exact keys (kSoft);
    // otherwise they serve groups whose top two keys are close and are read
    // from global memory, where they stay cached.
    __shared__ float2 tab_lds[kSoft ? kLogCells : 1];
    __shared__ float tile[kStage ? B * C : 2];
    const float2* tab = kSoft ? tab_lds : kLogCellTable.cell;
    if constexpr (kSoft) {
        fill_log_table(tab_lds);
        __syncthreads();
    }
    // The loop bound is uniform over the block (the tile copies are cooperative).
    for (int64_t base = (int64_t)blockIdx.x * B; base < a.ngroups; base += (int64_t)gridDim.x * B) {
        const int here = (int)(a.ngroups - base < B ? a.ngroups - base : B);
        const int64_t q = base + threadIdx.x;
        float alpha[C];
        if constexpr (kStage) {
            tile_in<B>(a.alpha + base * C, tile, here * C);
            __syncthreads();
            if ((int)threadIdx.x < here) {
#pragma unroll
                for (int c = 0; c < C; ++c) alpha[c] = tile[threadIdx.x * C + c];
            }
            __syncthreads(); // the tile is refilled next iteration
        }
        if ((int)threadIdx.x >= here) continue;
        if constexpr (!kStage) load_cat_logits<C>(a.alpha + q * C, alpha);
        uint32_t w[M];
        load_bf16<M>(a.W + q * M, w);
        uint32_t x[C];
        cat_words<C>(a.group0 + (uint64_t)q, a.key, x);
        float k[C];
        int best = 0;
        bool exact = true;
        if constexpr (!kSoft) {
            // hardware-log keys; decided when the top two are further apart
            // than the error margin of two keys (noise.hpp)
            // (scanned like the exact argmax: a NaN or infinite key leaves the
            // gap undefined or the margin infinite, so the exact keys decide)
#pragma unroll
            for (int c = 0; c < C; ++c) k[c] = fast_key_log2(alpha[c], a.key_c, x[c]);
            float top = k[0], second = -INFINITY, big = fabsf(k[0]);
#pragma unroll
            for (int c = 1; c < C; ++c) {
                big = fmaxf(big, fabsf(k[c]));
                const bool better = k[c] > top;
                second = better ? top : fmaxf(second, k[c]);
                best = better ? c : best;
                top = better ? k[c] : top;
            }
            const float margin = __builtin_fmaf(big, 0x1p-20f, kFastPairMargin);
            exact = C > 1 && !(top - second > margin);
        }
        if (exact) {
            cat_exact_keys<C>(alpha, x, a.lambda, tab, k);
            float top = k[0];
            best = 0;
#pragma unroll
            for (int c = 1; c < C; ++c) {
                const bool better = k[c] > top; // strict: ties keep the lower candidate
                best = better ? c : best;
                top = better ? k[c] : top;
            }
        }
        {
            uint32_t mask = 0;
#pragma unroll
            for (int c = 0; c < C; ++c) mask = best == c ? kCand<M, N>.mask[c] : mask;
            uint32_t out[M];
#pragma unroll
            for (int j = 0; j < M; ++j) out[j] = ((mask >> j) & 1u) ? w[j] : 0u;
            if constexpr (M == 4) {
                const u32x2 v = {out[0] | (out[1] << 16), out[2] | (out[3] << 16)};
                stream_store(v, reinterpret_cast<u32x2*>(a.Wm + q * M));
            } else {
                const u32x4 v = {out[0] | (out[1] << 16), out[2] | (out[3] << 16),
                                 out[4] | (out[5] << 16), out[6] | (out[7] << 16)};
                stream_store(v, reinterpret_cast<u32x4*>(a.Wm + q * M));
            }
            if (a.choice) stream_store((uint8_t)best, a.choice + q);
        }
        if constexpr (kSoft) {
            cat_softmax<C>(k, kLog2e * a.inv_tau);
            float S[M];
#pragma unroll
            for (int j = 0; j < M; ++j) S[j] = 0.0f;
#pragma unroll
            for (int c = 0; c < C; ++c) {
#pragma unroll
                for (int j = 0; j < M; ++j)
                    if ((kCand<M, N>.mask[c] >> j) & 1) S[j] += k[c];
            }
            if (a.S) store_f32<M>(a.S + q * M, S);
        }
    }
}

// The keys from the logits and the noise ng = -g of a group's candidates,
// kappa = fl(fl(alpha / lambda) + g); lambda = 1 is a wave-uniform branch
// without the division.
template <int C>
__device__ __forceinline__ void cat_keys_from_noise(const float (&alpha)[C], const float (&ng)[C],
                                                    float lambda, float (&k)[C])
{
    if (__builtin_amdgcn_readfirstlane(__float_as_uint(lambda)) == 0x3F800000u) {
#pragma unroll
        for (int c = 0; c < C; ++c) k[c] = alpha[c] - ng[c];
    } else {
#pragma unroll
        for (int c = 0; c < C; ++c) k[c] = alpha[c] / lambda - ng[c];
    }
}

// One chunk of B groups of the categorical backward.  The loads go out first:
// the group's W and dL/dW_masked, its logits (per lane, or for the staged
// tile this thread's share of the block's contiguous logits), and the log
// cells.  With up to 8 candidates the noise -- C Philox words and 2C
// logarithms per group, most of the arithmetic -- needs none of them and runs
// while they are in flight; with more, the C noise values and the tile share
// would not fit in registers beside each other, and each key is formed as its
// noise is drawn, after the loads.  kFull: all B groups are inside the
// array, so no per-lane condition makes the compiler wait for every load at
// a join.
template <int M, int N, bool kFull>
__device__ __forceinline__ void cat_bwd_chunk(const CatArgs& a, float* tile, float2* tab,
                                              int64_t base)
{
    constexpr int C = Candidates<M, N>::C;
    constexpr int B = cat_block(C);
    constexpr bool kStage = cat_staged_bwd(C);
    constexpr bool kNoiseFirst = C <= 8;
    constexpr int kShare = kStage && kNoiseFirst ? C / 2 : 1; // 8-byte tile pieces per thread
    const int here = kFull ? B : (int)(a.ngroups - base);
    const int64_t q = base + threadIdx.x;
    const bool live = kFull || (int)threadIdx.x < here;
    uint32_t w[M / 2], g[M / 2];
    float alpha[C];
    f32x2v share[kShare];
    if (live) {
        load_bf16_pairs<M>(a.W + q * M, w);
        load_bf16_pairs<M>(a.G + q * M, g);
    }
    if constexpr (kStage) {
        if constexpr (kFull && kNoiseFirst) {
            const f32x2v* src = reinterpret_cast<const f32x2v*>(a.alpha + base * C);
#pragma unroll
            for (int i = 0; i < kShare; ++i) share[i] = stream_load(src + threadIdx.x + i * B);
        }
    } else if (live) {
        load_cat_logits<C>(a.alpha + q * C, alpha);
    }
    const float4 cells = log_cells_of_lane();
    __builtin_amdgcn_sched_barrier(0);
    float ng[kNoiseFirst ? C : 1];
    uint32_t x[C];
    cat_words<C>(a.group0 + (uint64_t)q, a.key, x);
    publish_log_table(tab, cells);
    if constexpr (kNoiseFirst) {
#pragma unroll
        for (int c = 0; c < C; ++c) ng[c] = neg_gumbel_from_word(x[c], tab);
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (kStage) {
        if constexpr (kFull && kNoiseFirst) {
            f32x2v* dst = reinterpret_cast<f32x2v*>(tile);
#pragma unroll
            for (int i = 0; i < kShare; ++i) dst[threadIdx.x + i * B] = share[i];
        } else {
            tile_in<B>(a.alpha + base * C, tile, here * C);
        }
        __syncthreads();
        if (live) {
#pragma unroll
            for (int c = 0; c < C; ++c) alpha[c] = tile[threadIdx.x * C + c];
        }
        __syncthreads(); // the gradients go into the same tile
    }
    float d[C];
    if (live) {
        // the keys the forward sampled, and their softmax
        float y[C];
        if constexpr (kNoiseFirst)
            cat_keys_from_noise<C>(alpha, ng, a.lambda, y);
        else
            cat_exact_keys<C>(alpha, x, a.lambda, tab, y);
        cat_softmax<C>(y, kLog2e * a.inv_tau);
        // Straight-through: dL/dS = dL/dW_masked (.) W; ybar_c = sum_{j in c} sbar_j.
        float sbar[M];
#pragma unroll
        for (int i = 0; i < M / 2; ++i) {
            sbar[2 * i] = bf16_bits_to_float(g[i] & 0xFFFFu) * bf16_bits_to_float(w[i] & 0xFFFFu);
            sbar[2 * i + 1] = bf16_bits_to_float(g[i] >> 16) * bf16_bits_to_float(w[i] >> 16);
        }
        float ybar[C], dot = 0.0f;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            float acc = 0.0f;
#pragma unroll
            for (int j = 0; j < M; ++j)
                if ((kCand<M, N>.mask[c] >> j) & 1) acc += sbar[j];
            ybar[c] = acc;
            dot = __builtin_fmaf(y[c], acc, dot);
        }
        const float s = a.inv_tau * a.inv_lambda;
#pragma unroll
        for (int c = 0; c < C; ++c) d[c] = y[c] * (ybar[c] - dot) * s;
    }
    if constexpr (kStage) {
        if (live) {
#pragma unroll
            for (int c = 0; c < C; ++c) tile[threadIdx.x * C + c] = d[c];
        }
        __syncthreads();
        tile_out<B>(tile, a.dalpha + base * C, here * C);
        __syncthreads(); // before the next chunk overwrites the tile
    } else if (live) {
        store_cat<C>(a.dalpha + q * C, d);
    }
}

template <int M, int N>
__global__ __launch_bounds__(cat_block(Candidates<M, N>::C)) void cat_bwd_kernel(CatArgs a)
{
    constexpr int C = Candidates<M, N>::C;
    constexpr int B = cat_block(C);
    __shared__ float tile[cat_staged_bwd(C) ? B * C : 2];
    // Every group takes the exact keys; the block's waves share one copy of
    // the log cells in LDS (noise.hpp).
    __shared__ float4 tab4[kLogCells / 2];
    float2* tab = reinterpret_cast<float2*>(tab4);
    // The loop bound and the full / partial choice are uniform over the block
    // (the tile copies are cooperative).
    for (int64_t base = (int64_t)blockIdx.x * B; base < a.ngroups; base += (int64_t)gridDim.x * B) {
        if (base + B <= a.ngroups)
            cat_bwd_chunk<M, N, true>(a, tile, tab, base);
        else
            cat_bwd_chunk<M, N, false>(a, tile, tab, base);
    }
}

template <int M, int... Ns>
void* cat_fwd_for_n(int n, bool soft, std::integer_sequence<int, Ns...>)
{
    void* f = nullptr;
    ((n == Ns + 1 ? (f = soft ? (void*)cat_fwd_kernel<M, Ns + 1, true>
                              : (void*)cat_fwd_kernel<M, Ns + 1, false>,
                     0)
                  : 0),
     ...);
    return f;
}

template <int M, int... Ns>
void* cat_bwd_for_n(int n, std::integer_sequence<int, Ns...>)
{
    void* f = nullptr;
    ((n == Ns + 1 ? (f = (void*)cat_bwd_kernel<M, Ns + 1>, 0) : 0), ...);
    return f;
}

} // namespace
} // namespace roi

using namespace roi;

extern "C" int roi_cat_num_candidates(int n, int m)
{
    if ((m != 4 && m != 8) || n < 1 || n > m) return -1;
    return binom(m, n);
}

namespace roi {
namespace {
int cat_run(bool fwd, const uint16_t* W, const float* alpha, const uint16_t* G, int64_t rows,
            int64_t cols, int n, int m, float tau, float lambda, uint64_t seed, uint64_t step,
            uint64_t group_offset, uint16_t* W_masked, float* S, uint8_t* choice, float* dalpha,
            hipStream_t stream)
{
    const char* what = fwd ? "roi_cat_mask_fwd" : "roi_cat_mask_bwd";
    int64_t ngroups;
    int C;
    if (int st = validate_cat(fwd, W, alpha, G, rows, cols, n, m, tau, lambda, group_offset,
                              W_masked, S, choice, dalpha, &ngroups, &C))
        return st;
    if (ngroups == 0) return ok();
    void* fn = m == 4 ? (fwd ? cat_fwd_for_n<4>(n, S != nullptr, std::make_integer_sequence<int, 4>{})
                             : cat_bwd_for_n<4>(n, std::make_integer_sequence<int, 4>{}))
                      : (fwd ? cat_fwd_for_n<8>(n, S != nullptr, std::make_integer_sequence<int, 8>{})
                             : cat_bwd_for_n<8>(n, std::make_integer_sequence<int, 8>{}));
    if (!fn) return fail(ROI_E_UNSUPPORTED, "no kernel for %d:%d", n, m);
    CatArgs a{};
    a.W = W;
    a.alpha = alpha;
    a.G = G;
    a.Wm = W_masked;
    a.S = S;
    a.choice = choice;
    a.dalpha = dalpha;
    a.ngroups = ngroups;
    a.group0 = group_offset;
    a.key = make_key(seed, step, 0);
    a.lambda = lambda;
    a.key_c = (float)(1.4426950408889634 / (double)lambda);
    a.inv_lambda = (float)(1.0 / (double)lambda);
    a.inv_tau = (float)(1.0 / (double)tau);
    void* args[] = {&a};
    const int block = cat_block(C);
    if (hipLaunchKernel(fn, dim3(grid_for(ngroups, block)), dim3(block), args, 0, stream) !=
        hipSuccess)
        return launch_status(what);
    return launch_status(what);
}
} // namespace
} // namespace roi

extern "C" int roi_cat_mask_fwd(const uint16_t* W, const float* cat_logits, int64_t rows,
                                int64_t cols, int n, int m, float tau, float lambda, uint64_t seed,
                                uint64_t step, uint64_t group_offset, uint16_t* W_masked,
                                float* soft_mask, uint8_t* choice, hipStream_t stream)
{
    return cat_run(true, W, cat_logits, nullptr, rows, cols, n, m, tau, lambda, seed, step,
                   group_offset, W_masked, soft_mask, choice, nullptr, stream);
}

extern "C" int roi_cat_mask_bwd(const uint16_t* grad_W_masked, const uint16_t* W,
                                const float* cat_logits, int64_t rows, int64_t cols, int n, int m,
                                float tau, float lambda, uint64_t seed, uint64_t step,
                                uint64_t group_offset, float* grad_cat_logits, hipStream_t stream)
{
    return cat_run(false, W, cat_logits, grad_W_masked, rows, cols, n, m, tau, lambda, seed, step,
                   group_offset, nullptr, nullptr, nullptr, grad_cat_logits, stream);
}
