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
    uint32_t k0, k1;           // lo32 / hi32 of the seed
    uint32_t step_lo, step_hi; // counter words 2 and 3
    uint32_t block_hi;         // counter word 1: hi32 of the block index, the same for
                               // every element of one launch (launches are split where
                               // it changes)
};

__device__ __forceinline__ uint4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2,
                                               uint32_t c3, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)kPhiloxMul0 * (uint64_t)c0;
        const uint64_t p1 = (uint64_t)kPhiloxMul1 * (uint64_t)c2;
        // a ^ b ^ c in one gfx950 three-input bit operation (truth table 0x96)
        const uint32_t n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c1, k0, 0x96);
        const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c3, k1, 0x96);
        c1 = (uint32_t)p1;
        c3 = (uint32_t)p0;
        c0 = n0;
        c2 = n2;
        k0 += kWeyl0;
        k1 += kWeyl1;
    }
    return make_uint4(c0, c1, c2, c3);
}

// The four words for global elements 4*block .. 4*block+3; block_lo is the
// low 32 bits of the block index (the high 32 bits are key.block_hi).
// Counter words 1..3 are uniform over the launch, so the first two rounds
// run partly on the scalar unit.
__device__ __forceinline__ uint4 philox_block(uint32_t block_lo, const NoiseKey& key)
{
    return philox4x32_10(block_lo, key.block_hi, key.step_lo, key.step_hi, key.k0, key.k1);
}

// u = (2 (x >> 9) + 1) 2^-24: odd points of the 2^-24 grid, in (0, 1).
// Evaluated as (1 + (x >> 9) 2^-23) - (1 - 2^-24): the first term is the
// float with mantissa x >> 9 (one funnel shift of 0x7F:x by 9), and the
// difference is exact.
__device__ __forceinline__ float uniform_from_word(uint32_t x)
{
    return __uint_as_float(__builtin_amdgcn_alignbit(0x7Fu, x, 9)) - 0x1.fffffep-1f;
}

// Deterministic fp32 natural logarithm for finite normal x > 0, table-driven
// in the manner of Tang (ACM TOMS 1990):
//   x = z 2^k, z in [0.703125, 1.40625) (bit manipulation, exact);
//   z falls in one of 128 cells (76 of width 2^-8 below 1, 52 of width 2^-7
//   from 1 up); cell i holds inv_i = fl32(1/c_i) for its centre c_i and
//   lg_i = fl32(-ln inv_i), except the two cells touching 1, which hold
//   inv = 1 and lg = 0 so that r = z - 1 is exact there;
//   r = fma(z, inv_i, -1), ln(1 + r) ~ r + r^2 (-1/2 + r (1/3 - r/4));
//   ln x = k ln2 + lg_i + ln(1 + r).
// The cell constants come from a 15-term fp64 atanh series rounded to fp32.
// Every fp32 step is one IEEE operation in the order written (the library is
// compiled with -ffp-contract=off), so the value is reproducible bit for bit.
constexpr int kLogCells = 128;
constexpr int kLogCellsBelowOne = 76;
constexpr uint32_t kLogZBaseBits = 0x3F340000u; // 0.703125
constexpr float kLn2f = (float)0.69314718055994530941723212145818;
constexpr float kThird = (float)(1.0 / 3.0);

// fp64 ln by the atanh series, for the cell constants.
constexpr double ln_atanh_series(double v)
{
    const double s = (v - 1.0) / (v + 1.0);
    const double s2 = s * s;
    double acc = 0.0;
    for (int j = 14; j >= 0; --j) acc = acc * s2 + 2.0 / (double)(2 * j + 1);
    return s * acc;
}

// The cells in reverse order: entry j holds (inv, lg) of cell 127 - j, the
// order in which det_log_bits() indexes them.
struct alignas(16) LogCells {
    float2 cell[kLogCells];
};

// The cell constants, evaluated by the compiler (IEEE fp64, round to nearest).
constexpr LogCells make_log_cells()
{
    LogCells t{};
    for (int i = 0; i < kLogCells; ++i) {
        double lo = 0.0, width = 0.0;
        if (i < kLogCellsBelowOne) {
            lo = 0.703125 + (double)i / 256.0;
            width = 1.0 / 256.0;
        } else {
            lo = 1.0 + (double)(i - kLogCellsBelowOne) / 128.0;
            width = 1.0 / 128.0;
        }
        const double centre = lo + width / 2.0;
        float inv = 1.0f, lg = 0.0f;
        if (i != kLogCellsBelowOne - 1 && i != kLogCellsBelowOne) {
            inv = (float)(1.0 / centre);
            lg = (float)(-ln_atanh_series((double)inv));
        }
        t.cell[kLogCells - 1 - i].x = inv;
        t.cell[kLogCells - 1 - i].y = lg;
    }
    return t;
}

static __device__ const LogCells kLogCellTable = make_log_cells();

// Copies the cells into the block's LDS copy; threads 0..127 each copy one.
// The caller synchronises the block before the first lookup.
__device__ __forceinline__ void fill_log_table(float2* tab)
{
    const int i = threadIdx.x;
    if (i < kLogCells) tab[i] = kLogCellTable.cell[i];
}

// The cells in LDS for kernels in which every group takes the exact keys:
// one 1 KiB copy per block.  Lane l holds cells 2l and 2l + 1 (16 bytes),
// loaded with log_cells_of_lane() ahead of the kernel's HBM streams, so that
// waiting for this cached read does not wait for them.  Every wave then
// stores the whole table with publish_log_table(): the same values at the
// same addresses, so a wave whose own writes have completed (lgkmcnt 0) sees
// the cells whatever the other waves do, and no wave waits for another (no
// block barrier).  Every lane of the wave must take part.
__device__ __forceinline__ float4 log_cells_of_lane()
{
    // The empty asm keeps the load where it is written (inside the caller's
    // loop): hoisted out of the loop, its four registers would stay live
    // through the whole loop body.
    int lane = (int)(threadIdx.x & 63);
    asm volatile("" : "+v"(lane));
    return reinterpret_cast<const float4*>(kLogCellTable.cell)[lane];
}

__device__ __forceinline__ void publish_log_table(float2* tab, float4 cells)
{
    reinterpret_cast<float4*>(tab)[threadIdx.x & 63] = cells;
    __builtin_amdgcn_s_waitcnt(0xC07F); // lgkmcnt(0); vmcnt and expcnt not waited for
    __builtin_amdgcn_wave_barrier();
}

// ln of the float whose bit pattern is ix.  With t = ix - kLogZBaseBits the
// exponent is k = floor(t / 2^23), z = x 2^-k and the cell is bits 16..22 of
// t.  The code forms v = 0x7FFFFF - t instead: its low 23 bits are those of t
// complemented and -k = floor(v / 2^23), so v gives -k by one shift, the cell
// by its bits 16..22 (counted from the top, hence the reversed table), and z
// as ix + (-k) 2^23.  fma(-k, -ln 2, s) equals fma(k, ln 2, s).
__device__ __forceinline__ float det_log_bits(uint32_t ix, const float2* tab)
{
    const uint32_t v = (0x7FFFFFu + kLogZBaseBits) - ix;
    int nk = (int)v >> 23;
    // Hides that nk came from v: the compiler would otherwise fold the shifts
    // into a mask and an add, one instruction more than the shift-add.
    asm("" : "+v"(nk));
    const float z = __uint_as_float(ix + ((uint32_t)nk << 23));
    const float2 c = tab[(v >> 16) & 0x7Fu];
    const float r = __builtin_fmaf(z, c.x, -1.0f);
    float p = __builtin_fmaf(r, -0.25f, kThird);
    p = __builtin_fmaf(r, p, -0.5f);
    const float r2 = r * r;
    const float l1p = __builtin_fmaf(r2, p, r);
    const float s = c.y + l1p;
    return __builtin_fmaf((float)nk, -kLn2f, s);
}

__device__ __forceinline__ float det_log(float x, const float2* tab)
{
    return det_log_bits(__float_as_uint(x), tab);
}

// Returns ln(-ln u) = -g for the Gumbel noise g = -log(-log u).  ln u < 0 for
// every u < 1, so the bits of -ln u are those of ln u minus the sign bit.
__device__ __forceinline__ float neg_gumbel_from_word(uint32_t x, const float2* tab)
{
    const float u = uniform_from_word(x);
    const float lu = det_log(u, tab);
    return det_log_bits(__float_as_uint(lu) - 0x80000000u, tab);
}

__device__ __forceinline__ float gumbel_from_word(uint32_t x, const float2* tab)
{
    return -neg_gumbel_from_word(x, tab);
}

// Keys from the hardware logarithm (v_log_f32), in log2 units.
//
// The noise: N(x) = -log2(-log2 u(x)), which approximates g log2(e) + log2(ln 2)
// for the g of neg_gumbel_from_word.  Over every one of the 2^23 possible u
// its distance from that value, with g the library's own fp32 noise, is below
// kFastNoiseBound (the largest is 1.98e-6, at u close to 1, where |N| ~ 23).
// The common offset log2(ln 2) cancels in every comparison and softmax.
//
// The key: K = fma(phi, c, N(x)) with c = fl(log2(e) / lambda), which
// approximates log2(e) kappa + log2(ln 2) for kappa = fl(fl(phi / lambda) + g).
// With a = fl(phi / lambda), |g| < 16.7 and |a| <= |kappa| + |g| the error is
// at most
//   kFastNoiseBound                      the noise
//   + 3 * 2^-24 log2(e) |a|              c and a each round once
//   + 2^-24 log2(e) |kappa|              the rounding of kappa
//   + 2^-24 |K|                          the rounding of the fma
//   <= 6.9e-6 + 2.98e-7 |K|              (log2(e) |kappa| <= |K| + 0.54).
// Two keys i, j whose hardware keys differ by more than
//   kFastPairMargin + 2^-20 max(|K_i|, |K_j|) > the sum of the two errors
// are therefore ordered the same way by kappa, and are not equal.  These keys
// serve comparisons only: the straight-through forward ranks with them and
// recomputes the exact keys for any group in which two keys are closer than
// the margin, so its selections are those of the exact keys.  Every
// relaxation (the soft mask, the soft forward and every backward) runs at the
// exact keys.
constexpr float kFastNoiseBound = 2.5e-6f;
constexpr float kFastPairMargin = 3.2e-5f; // > 2 (kFastNoiseBound + 4.44e-6), with slack

__device__ __forceinline__ float fast_noise_log2(uint32_t x)
{
    const float u = uniform_from_word(x);
    const float l1 = __builtin_amdgcn_logf(u); // log2 u < 0
    return -__builtin_amdgcn_logf(-l1);
}

__device__ __forceinline__ float fast_key_log2(float phi, float c, uint32_t x)
{
    return __builtin_fmaf(phi, c, fast_noise_log2(x));
}

// True when every pair of the m hardware keys is further apart than the
// margin above, taken with the group's largest |K| (which only widens it);
// false whenever a key is infinite or NaN.
template <int M>
__device__ __forceinline__ bool fast_keys_separated(const float (&k)[M])
{
    float big = fabsf(k[0]);
#pragma unroll
    for (int j = 1; j < M; ++j) big = fmaxf(big, fabsf(k[j]));
    const float margin = __builtin_fmaf(big, 0x1p-20f, kFastPairMargin);
    bool sep = true;
#pragma unroll
    for (int i = 0; i < M; ++i) {
#pragma unroll
        for (int j = i + 1; j < M; ++j) sep &= fabsf(k[i] - k[j]) > margin;
    }
    return sep;
}

// phi / lambda for the four elements of a slot, correctly rounded; lambda == 1
// (wave-uniform) takes phi as it is.  The division is a separate branch on
// purpose: a select between phi and the quotient would run the division's
// whole IEEE sequence at lambda = 1 too.
__device__ __forceinline__ void scaled_logits4(const float (&phi)[4], float lambda, float (&a)[4])
{
    if (__builtin_amdgcn_readfirstlane(__float_as_uint(lambda)) == 0x3F800000u) {
#pragma unroll
        for (int e = 0; e < 4; ++e) a[e] = phi[e];
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) a[e] = phi[e] / lambda;
    }
}

// kappa = fl(fl(phi / lambda) + g); for lambda == 1 the quotient is phi exactly.
template <bool kLambdaOne>
__device__ __forceinline__ float key_of(float phi, float lambda, uint32_t word, const float2* tab)
{
    const float ng = neg_gumbel_from_word(word, tab);
    const float phi_bar = kLambdaOne ? phi : phi / lambda;
    return phi_bar - ng;
}

} // namespace roi
