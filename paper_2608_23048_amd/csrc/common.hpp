// common.hpp -- pieces shared by the kernels of the RoI sampler: launch
// geometry, the argument blocks, and the HBM stream loads and stores.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "noise.hpp"

namespace roi {

constexpr int kBlock = 256;

// Non-temporal hints on the HBM streams (each byte is touched once).
#ifndef ROI_NONTEMPORAL
#define ROI_NONTEMPORAL 1
#endif

struct FwdArgs {
    const uint16_t* W;
    const float* phi;
    uint16_t* Wm;
    float* S;
    uint8_t* idx;
    int64_t ngroups;
    uint32_t block0; // low 32 bits of elem_offset / 4 (the high 32 are key.block_hi)
    NoiseKey key;
    float lambda;
    float key_c; // fl(log2(e) / lambda): the scale of the hardware-log keys
    float inv_tau;
    int soft; // 1: W_masked = W (.) S (pure soft forward), 0: W (.) hard mask
};

struct BwdArgs {
    const uint16_t* G;
    const uint16_t* W;
    const float* phi;
    float* dphi;
    int64_t ngroups;
    uint32_t block0;
    NoiseKey key;
    float key_c; // fl(log2(e) / lambda)
    float inv_lambda;
    float tau;
    float inv_tau;
};

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename T>
__device__ __forceinline__ T stream_load(const T* p)
{
#if ROI_NONTEMPORAL
    return __builtin_nontemporal_load(p);
#else
    return *p;
#endif
}

template <typename T>
__device__ __forceinline__ void stream_store(const T& v, T* p)
{
#if ROI_NONTEMPORAL
    __builtin_nontemporal_store(v, p);
#else
    *p = v;
#endif
}

__device__ __forceinline__ float bf16_bits_to_float(uint32_t b) { return __uint_as_float(b << 16); }

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t float_to_bf16_rne(float f)
{
    const uint32_t b = __float_as_uint(f);
    return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

// Loads of one group: m fp32 logits (m/4 16-byte loads) and m bf16 values
// (one 8-byte load for m = 4, one 16-byte load for m = 8).
template <int M>
__device__ __forceinline__ void load_logits(const float* p, float (&phi)[M])
{
    const f32x4* p4 = reinterpret_cast<const f32x4*>(p);
#pragma unroll
    for (int t = 0; t < M / 4; ++t) {
        const f32x4 v = stream_load(p4 + t);
        phi[4 * t + 0] = v.x;
        phi[4 * t + 1] = v.y;
        phi[4 * t + 2] = v.z;
        phi[4 * t + 3] = v.w;
    }
}

template <int M>
__device__ __forceinline__ void load_bf16(const uint16_t* p, uint32_t (&w)[M])
{
    if constexpr (M == 4) {
        const u32x2 v = stream_load(reinterpret_cast<const u32x2*>(p));
        w[0] = v.x & 0xFFFFu; w[1] = v.x >> 16; w[2] = v.y & 0xFFFFu; w[3] = v.y >> 16;
    } else {
        static_assert(M == 8, "m");
        const u32x4 v = stream_load(reinterpret_cast<const u32x4*>(p));
        w[0] = v.x & 0xFFFFu; w[1] = v.x >> 16; w[2] = v.y & 0xFFFFu; w[3] = v.y >> 16;
        w[4] = v.z & 0xFFFFu; w[5] = v.z >> 16; w[6] = v.w & 0xFFFFu; w[7] = v.w >> 16;
    }
}

using FwdFn = void (*)(FwdArgs);
using BwdFn = void (*)(BwdArgs);

// Kernels for m = 16 and 32 (wide.hip): four consecutive elements per lane,
// a group spread over m / 4 adjacent lanes.
FwdFn select_wide_fwd(int m, int n);
BwdFn select_wide_bwd(int m, int n);

} // namespace roi
