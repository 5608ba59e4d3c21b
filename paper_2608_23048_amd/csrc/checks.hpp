// checks.hpp -- the library's host-side argument checks.  Plain C++ with no
// GPU code, so that the same file also builds with the host compiler alone
// (and its address and undefined-behaviour sanitizers).  Every entry point of
// the C ABI runs these before it launches anything; a failure returns a
// status and leaves its detail in the thread-local error text.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "roi.h"

namespace roi {

// Thread-local detail of the last failure (returned by roi_last_error).
extern thread_local std::string g_last_error;

// Records a printf-style detail and returns `status`.
int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Clears the detail and returns ROI_OK.
int ok();
bool aligned16(const void* p);
// Whether [a, a + na) and [b, b + nb) share a byte (empty ranges share none).
bool overlap(const void* a, size_t na, const void* b, size_t nb);

// One checked address range of a call: [p, p + n), an input or an output.
struct Range {
    uintptr_t p;
    size_t n;
    bool out;
};
// Fails when an output overlaps any other range (inputs may overlap inputs).
int check_overlaps(std::vector<Range>& r);
void add_range(std::vector<Range>& r, const void* p, size_t n, bool out);

// The sizes of one [rows, cols] tensor of groups of m.
struct Shape {
    int64_t numel = 0;
    int64_t ngroups = 0;
};
// Pattern (1 <= n <= m, m in {4, 8, 16, 32}), finite positive temperatures.
int check_common(int n, int m, float tau, float lambda);
// check_common plus the tensor's sizes and its global element offset.
int check_shape(int64_t rows, int64_t cols, int n, int m, float tau, float lambda,
                uint64_t elem_offset, Shape* sh);
// A descriptor array of `count` entries (NULL only when empty).
int check_count(const void* t, int count);

// One AdamW step folded into constants (host, fp64, rounded once):
// phi <- phi * decay - step_size * m' / (sqrt(v') * inv_sqrt_bc2 + eps),
// m' = beta1 m + (1 - beta1) g, v' = beta2 v + (1 - beta2) g^2.
struct AdamStep {
    float decay;        // 1 - lr * weight_decay
    float beta1, beta2;
    float one_m_beta1, one_m_beta2;
    float step_size;    // lr / (1 - beta1^t)
    float inv_sqrt_bc2; // 1 / sqrt(1 - beta2^t)
    float eps;
};
int check_adamw(const roi_adamw_params* o, AdamStep* st);

// The forward's tensors: sets *with_s / *with_idx to whether the soft mask and
// the indices are requested (-1 when every tensor is empty: nothing to do).
int validate_fwd(const roi_fwd_tensor* t, int count, int n, int m, float tau, float lambda,
                 int* with_s, int* with_idx);

// One tensor of a backward call; phi is overwritten with the updated logits
// when the AdamW step is fused (m and v set).
struct BwdDesc {
    const uint16_t* G;
    const uint16_t* W;
    const float* phi;
    float* dphi;
    float* m;
    float* v;
    int64_t rows, cols;
    uint64_t off;
};
// The backward's tensors (opt: the fused AdamW step or NULL, folded into *st);
// *any is false when every tensor is empty.
int validate_bwd(const BwdDesc* t, int count, int n, int m, float tau, float lambda,
                 const roi_adamw_params* opt, AdamStep* st, bool* any);

// The categorical sampler's arguments (m in {4, 8}): sets the group count and
// the number of candidates C = binom(m, n) per group.
int validate_cat(bool fwd, const uint16_t* W, const float* alpha, const uint16_t* G, int64_t rows,
                 int64_t cols, int n, int m, float tau, float lambda, uint64_t group_offset,
                 const uint16_t* W_masked, const float* S, const uint8_t* choice,
                 const float* dalpha, int64_t* ngroups, int* C);

// Calls launch(first, count, elem0) for consecutive pieces of [0, items) --
// items of `per_item` elements starting at global element elem_offset -- so
// that within a piece every Philox block index (element / 4) has the same high
// 32 bits.  Pieces end at multiples of 2^34 elements, which per_item divides.
template <typename F>
int for_each_piece(uint64_t elem_offset, int64_t items, int64_t per_item, F&& launch)
{
    int64_t done = 0;
    while (done < items) {
        const uint64_t e0 = elem_offset + (uint64_t)done * (uint64_t)per_item;
        const uint64_t boundary = ((e0 >> 34) + 1) << 34;
        const uint64_t fit = (boundary - e0) / (uint64_t)per_item;
        const int64_t left = items - done;
        const int64_t count = fit < (uint64_t)left ? (int64_t)fit : left;
        if (int st = launch(done, count, e0)) return st;
        done += count;
    }
    return ROI_OK;
}

} // namespace roi
