// host.hpp -- host-side helpers shared by the library's translation units:
// the thread-local error text, argument checks and launch geometry.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "common.hpp"
#include "noise.hpp"

namespace roi {

// Thread-local detail of the last failure (returned by roi_last_error).
extern thread_local std::string g_last_error;

// Records a printf-style detail and returns `status`.
int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Clears the detail and returns ROI_OK.
int ok();
bool aligned16(const void* p);
bool overlap(const void* a, size_t na, const void* b, size_t nb);
// One-shot grid for `items` threads (below 2^32 threads in total).
int grid_for(int64_t items, int block = kBlock);
// Philox key and step words of a call.
NoiseKey make_key(uint64_t seed, uint64_t step, uint64_t block);
// ROI_OK, or ROI_E_HIP with the runtime's error after a launch.
int launch_status(const char* what);

// One checked address range of a call: [p, p + n), an input or an output.
struct Range {
    uintptr_t p;
    size_t n;
    bool out;
};
// Fails when an output overlaps any other range (inputs may overlap inputs).
int check_overlaps(std::vector<Range>& r);
void add_range(std::vector<Range>& r, const void* p, size_t n, bool out);

} // namespace roi
