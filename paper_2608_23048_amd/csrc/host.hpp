// host.hpp -- host-side helpers shared by the library's translation units:
// the argument checks (checks.hpp) and launch geometry.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "checks.hpp"
#include "common.hpp"
#include "noise.hpp"

namespace roi {

// One-shot grid for `items` threads (below 2^32 threads in total).
int grid_for(int64_t items, int block = kBlock);
// Philox key and step words of a call.
NoiseKey make_key(uint64_t seed, uint64_t step, uint64_t block);
// ROI_OK, or ROI_E_HIP with the runtime's error after a launch.
int launch_status(const char* what);

} // namespace roi
