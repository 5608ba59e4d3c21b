// common.hpp -- pieces shared by the kernels of the RoI sampler: launch
// geometry, the argument blocks, and the HBM stream loads and stores.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "checks.hpp"
#include "noise.hpp"

namespace roi {

constexpr int kBlock = 256;

// Non-temporal hints on the HBM streams (each byte is touched once).
#ifndef ROI_NONTEMPORAL
#define ROI_NONTEMPORAL 1
#endif

// A launch processes a batch of up to kMaxPieces pieces: consecutive groups of
// one tensor whose Philox block indices share their high 32 bits.  Piece i
// owns the launch's blocks [first_block, first_block + nblocks); its blocks
// stride over the piece when it has more groups than blocks cover.
constexpr int kMaxPieces = 32;
static_assert((kMaxPieces & (kMaxPieces - 1)) == 0, "binary search over the pieces");

struct FwdPiece {
    const uint16_t* W;
    const float* phi;
    uint16_t* Wm;
    float* S;
    uint8_t* idx;
    int64_t ngroups;
    uint32_t block0;   // low 32 bits of the Philox block index (element / 4) of group 0
    uint32_t block_hi; // its high 32 bits, the same for every group of the piece
    uint32_t first_block, nblocks;
};

// starts[i]: the first block of piece i (= p[i].first_block), and 0xFFFFFFFF
// for the unused entries, contiguous so that a block finds its piece from two
// wide scalar loads.
struct FwdBatch {
    uint32_t starts[kMaxPieces];
    FwdPiece p[kMaxPieces];
    int count;
    NoiseKey key_base; // key_base.block_hi is replaced by the piece's
    float lambda;
    float key_c; // fl(log2(e) / lambda): the scale of the hardware-log keys
    float inv_tau;
    float key_scale; // fl(fl(log2(e)) * inv_tau): exact keys to softmax arguments in log2 units
    float exp_span; // key-span limit of the exp-domain relaxation (relax.hpp)
    int soft; // 1: W_masked = W (.) S (pure soft forward), 0: W (.) hard mask
};

struct BwdPiece {
    const uint16_t* G;
    const uint16_t* W;
    const float* phi;
    float* dphi;   // dL/dphi (may be NULL when the optimizer step is fused)
    float* m;      // AdamW first and second moments (fused optimizer step only);
    float* v;      // the updated logits are written over phi
    int64_t ngroups;
    uint32_t block0, block_hi;
    uint32_t first_block, nblocks;
};

struct BwdBatch {
    uint32_t starts[kMaxPieces]; // as in FwdBatch
    BwdPiece p[kMaxPieces];
    int count;
    NoiseKey key_base; // key_base.block_hi is replaced by the piece's
    float lambda;
    float inv_lambda;
    float tau;
    float inv_tau;
    float key_scale; // fl(fl(log2(e)) * inv_tau), as in FwdBatch
    float exp_span; // key-span limit of the exp-domain relaxation (relax.hpp)
    AdamStep adam;
};

// A batch travels as the kernel's argument block, which is at most 4 KiB.
static_assert(sizeof(FwdBatch) <= 4096 && sizeof(BwdBatch) <= 4096, "kernel arguments");

// The fused AdamW update of one logit from its gradient g (fp32, fast
// reciprocal and square root: the result is held to the float tolerance).
__device__ __forceinline__ void adamw_update(const AdamStep& a, float g, float& phi, float& m,
                                             float& v)
{
    m = __builtin_fmaf(a.beta1, m, a.one_m_beta1 * g);
    v = __builtin_fmaf(a.beta2, v, a.one_m_beta2 * (g * g));
    const float den = __builtin_fmaf(__builtin_amdgcn_sqrtf(v), a.inv_sqrt_bc2, a.eps);
    phi = __builtin_fmaf(-a.step_size * m, __builtin_amdgcn_rcpf(den), phi * a.decay);
}

// The piece that owns this block: the last piece that starts at or before it,
// by binary search over the starts (unused entries are 0xFFFFFFFF).  Every
// wave of every block runs this on the CU's shared scalar unit, and a launch
// has millions of blocks of a few microseconds each, so it is kept to a few
// scalar instructions: none for a single piece, five steps otherwise.
template <typename Batch>
__device__ __forceinline__ int find_piece(const Batch& a)
{
    if (a.count == 1) return 0;
    const uint32_t b = blockIdx.x;
    int i = 0;
#pragma unroll
    for (int step = kMaxPieces / 2; step >= 1; step /= 2)
        if (b >= a.starts[i + step]) i += step;
    return i;
}

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

// The bf16 values nearest to lo and hi (ties to even), packed with lo in the
// low half: one gfx950 v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi)
{
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    const f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// bf16(W (.) S) for four consecutive elements: w holds the bf16 patterns of W
// in pairs (element 2i in the low half of w[i]).
__device__ __forceinline__ u32x2 soft_product4(uint32_t w01, uint32_t w23, const float* S)
{
    return u32x2{bf16x2_rne(bf16_bits_to_float(w01 & 0xFFFFu) * S[0],
                            bf16_bits_to_float(w01 >> 16) * S[1]),
                 bf16x2_rne(bf16_bits_to_float(w23 & 0xFFFFu) * S[2],
                            bf16_bits_to_float(w23 >> 16) * S[3])};
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

// The same loads, the values left in pairs (element 2i in the low half of
// word i).
template <int M>
__device__ __forceinline__ void load_bf16_pairs(const uint16_t* p, uint32_t (&w)[M / 2])
{
    if constexpr (M == 4) {
        const u32x2 v = stream_load(reinterpret_cast<const u32x2*>(p));
        w[0] = v.x; w[1] = v.y;
    } else {
        static_assert(M == 8, "m");
        const u32x4 v = stream_load(reinterpret_cast<const u32x4*>(p));
        w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    }
}

// m fp32 values of a group, stored as m/4 16-byte vectors.
template <int M>
__device__ __forceinline__ void store_f32(float* p, const float (&x)[M])
{
    f32x4* p4 = reinterpret_cast<f32x4*>(p);
#pragma unroll
    for (int t = 0; t < M / 4; ++t) {
        const f32x4 v = {x[4 * t], x[4 * t + 1], x[4 * t + 2], x[4 * t + 3]};
        stream_store(v, p4 + t);
    }
}

// The backward's inputs for four consecutive elements (one group of 4, or a
// lane's part of a wider group), as loaded: bf16 pairs stay packed.
template <bool kAdam>
struct BwdSlot {
    f32x4 phi;
    u32x2 w, g;
    f32x4 mom, sec; // AdamW moments (fused optimizer step only)
};

// Loads the slot of elements 4 s .. 4 s + 3 of a piece.
template <bool kAdam>
__device__ __forceinline__ void load_bwd_slot(const BwdPiece& pc, int64_t s, BwdSlot<kAdam>& in)
{
    in.phi = stream_load(reinterpret_cast<const f32x4*>(pc.phi + s * 4));
    in.w = stream_load(reinterpret_cast<const u32x2*>(pc.W + s * 4));
    in.g = stream_load(reinterpret_cast<const u32x2*>(pc.G + s * 4));
    if constexpr (kAdam) {
        in.mom = stream_load(reinterpret_cast<const f32x4*>(pc.m + s * 4));
        in.sec = stream_load(reinterpret_cast<const f32x4*>(pc.v + s * 4));
    }
}

using FwdFn = void (*)(FwdBatch);
using BwdFn = void (*)(BwdBatch);

// Final-mask export (export.hip): top-n of the logits of each group.
struct ExportArgs {
    const float* phi;
    const uint16_t* W;
    uint16_t* Wm;   // dense masked weights or NULL
    uint16_t* vals; // [groups, n] kept weights, increasing index, or NULL
    uint8_t* idx;   // [groups, n] their indices, or NULL
    uint32_t* meta; // [ceil(groups / 8)] 2:4 index fields, or NULL
    int64_t ngroups;
};
using ExportFn = void (*)(ExportArgs);
ExportFn select_export(int m, int n);

// Kernels for m = 16 and 32 (wide_fwd.hip, wide_bwd.hip): four consecutive elements per lane,
// a group spread over m / 4 adjacent lanes.
FwdFn select_wide_fwd(int m, int n, bool relax, int q); // q: tau_mode (roi.hip)
FwdFn select_wide_soft_only(int m, int n, int q);
BwdFn select_wide_bwd(int m, int n, bool adam, int q);
// Slots (four elements each) one block of the wide backward covers.
int64_t wide_bwd_block_slots(int m);

} // namespace roi
