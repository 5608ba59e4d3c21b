// stream_copy.hip -- a plain streaming copy on gfx950: the data-movement
// reference the benchmark sets beside the sampler's kernels.  It moves bytes
// the way they do (16 bytes per lane, non-temporal loads and stores, a
// one-shot grid of 256-thread blocks dispatched in address order), so its
// rate is what HBM delivers to that access pattern on the same GPU.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.hpp"
#include "host.hpp"
#include "roi.h"

namespace roi {
namespace {

__global__ __launch_bounds__(kBlock) void stream_copy_kernel(const u32x4* src, u32x4* dst,
                                                             int64_t count)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < count; i += stride)
        stream_store(stream_load(src + i), dst + i);
}

} // namespace
} // namespace roi

using namespace roi;

extern "C" int roi_stream_copy(const void* src, void* dst, int64_t nbytes, hipStream_t stream)
{
    if (nbytes < 0 || nbytes % 16 != 0)
        return fail(ROI_E_INVAL, "nbytes must be a non-negative multiple of 16 (got %lld)",
                    (long long)nbytes);
    if (nbytes == 0) return ok();
    if (!src || !dst) return fail(ROI_E_INVAL, "src and dst must not be NULL");
    if (!aligned16(src) || !aligned16(dst))
        return fail(ROI_E_INVAL, "device pointers must be 16-byte aligned");
    if (overlap(src, (size_t)nbytes, dst, (size_t)nbytes))
        return fail(ROI_E_INVAL, "src and dst overlap");
    const int64_t count = nbytes / 16;
    hipLaunchKernelGGL(stream_copy_kernel, dim3(grid_for(count)), dim3(kBlock), 0, stream,
                       static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), count);
    return launch_status("roi_stream_copy");
}
