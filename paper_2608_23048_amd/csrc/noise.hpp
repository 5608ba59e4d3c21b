// noise.hpp -- device-side noise of the RoI sampler for gfx950.
//
// Algorithm 1 (appendix) draws u ~ Uniform(0,1) and forms the Gumbel noise
// g = -log(-log u); §3.2 / §4.2.2 add it to the (scaled, §4.2.3) logits to get
// the keys.  Here u comes from a counter-based generator so that the backward
// can regenerate the forward's keys instead of storing them, and the
// logarithm is a fixed sequence of IEEE fp32 operations so that the keys are
// one reproducible fp32 value per (seed, step, element, logit).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace roi {

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): per round, the products
// of counter words 0 and 2 with the two Philox multipliers; the high halves
// are xor-ed with words 1 and 3 and the round key, the low halves move into
// words 1 and 3.  The key advances by the Weyl increments (golden ratio and
// sqrt(3) - 1 in 0.32 fixed point) after every round.
constexpr uint32_t kPhiloxMul0 = 0xD2511F53u;
constexpr uint32_t kPhiloxMul1 = 0xCD9E8D57u;
constexpr uint32_t kWeyl0 = 0x9E3779B9u;
constexpr uint32_t kWeyl1 = 0xBB67AE85u;

struct NoiseKey {
    uint32_t k0, k1;          // lo32 / hi32 of the seed
    uint32_t step_lo, step_hi; // counter words 2 and 3
};

__device__ __forceinline__ uint4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2,
                                               uint32_t c3, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)kPhiloxMul0 * (uint64_t)c0;
        const uint64_t p1 = (uint64_t)kPhiloxMul1 * (uint64_t)c2;
        const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        c1 = (uint32_t)p1;
        c3 = (uint32_t)p0;
        c0 = n0;
        c2 = n2;
        k0 += kWeyl0;
        k1 += kWeyl1;
    }
    return make_uint4(c0, c1, c2, c3);
}

// The four words for global elements 4*block .. 4*block+3.
__device__ __forceinline__ uint4 philox_block(uint64_t block, const NoiseKey& key)
{
    return philox4x32_10((uint32_t)block, (uint32_t)(block >> 32), key.step_lo, key.step_hi,
                         key.k0, key.k1);
}

// u = (2 (x >> 9) + 1) 2^-24: odd points of the 2^-24 grid, in (0, 1), exact.
__device__ __forceinline__ float uniform_from_word(uint32_t x)
{
    return (float)(((x >> 9) << 1) | 1u) * 0x1p-24f;
}

// Deterministic fp32 natural logarithm for finite normal x > 0.
// x = m 2^E with m in [sqrt(1/2), sqrt(2)); ln m = 2 atanh(s), s = f / (f + 2),
// f = m - 1 (exact), summed as 2s + s^3 (2/3 + 2/5 s^2 + 2/7 s^4 + 2/9 s^6);
// ln 2 is split into a 16-bit head (E * head is exact) and an fp32 tail.
// Each line below is one correctly rounded fp32 operation; the file is
// compiled with -ffp-contract=off so none is fused or reordered, and '/' is
// the IEEE division.
constexpr double kLn2 = 0.69314718055994530941723212145818;
constexpr float kLn2Head = (float)(45426.0 / 65536.0); // ln 2 truncated to 16 bits
constexpr float kLn2Tail = (float)(kLn2 - 45426.0 / 65536.0);
constexpr float kAtanh3 = (float)(2.0 / 3.0);
constexpr float kAtanh5 = (float)(2.0 / 5.0);
constexpr float kAtanh7 = (float)(2.0 / 7.0);
constexpr float kAtanh9 = (float)(2.0 / 9.0);
static_assert(45426.0 / 65536.0 <= kLn2 && kLn2 < 45427.0 / 65536.0, "ln2 head");

__device__ __forceinline__ float det_log(float x)
{
    const uint32_t bits = __float_as_uint(x);
    int e = (int)(bits >> 23) - 127;
    const uint32_t mbits = (bits & 0x7FFFFFu) | 0x3F800000u; // m in [1, 2)
    float m = __uint_as_float(mbits);
    if (mbits >= 0x3FB504F4u) { // m > sqrt(2): use m/2 and E+1
        m = m * 0.5f;
        e = e + 1;
    }
    const float f = m - 1.0f;
    const float s = f / (f + 2.0f);
    const float z = s * s;
    float p = __builtin_fmaf(kAtanh9, z, kAtanh7);
    p = __builtin_fmaf(p, z, kAtanh5);
    p = __builtin_fmaf(p, z, kAtanh3);
    const float t = s * z;
    const float r = __builtin_fmaf(t, p, s + s);
    const float ef = (float)e;
    const float lo = __builtin_fmaf(ef, kLn2Tail, r);
    return __builtin_fmaf(ef, kLn2Head, lo);
}

// g = -log(-log u)
__device__ __forceinline__ float gumbel_from_word(uint32_t x)
{
    const float u = uniform_from_word(x);
    const float y = -det_log(u);
    return -det_log(y);
}

// kappa = fl(fl(phi / lambda) + g); for lambda == 1 the quotient is phi exactly.
template <bool kLambdaOne>
__device__ __forceinline__ float key_of(float phi, float lambda, uint32_t word)
{
    const float g = gumbel_from_word(word);
    const float phi_bar = kLambdaOne ? phi : phi / lambda;
    return phi_bar + g;
}

} // namespace roi
