// sparse_mfma_check.hip -- test-side consumer of the 2:4 export: a plain
// sparse-MFMA product Y = W_sparse X^T on gfx950, fed directly by the
// compressed values and metadata that roi_mask_export writes.  It exists to
// show that the export's layout is the one the matrix core reads; it is not
// part of the library.
//
// v_smfmac_f32_16x16x64_bf16 (one wave, a 16 x 64 2:4-sparse A tile, a 64 x 16
// B tile, a 16 x 16 fp32 accumulator), operand layout as measured on gfx950:
//   A  lane l holds row l % 16, compressed columns 8 (l / 16) .. + 7, which
//      cover the dense columns 16 (l / 16) .. + 15 (two kept values per group
//      of four, lower index first);
//   idx lane l: 4 bits per group of four, group p of the lane's 16 columns in
//      bits 4p .. 4p + 3, the lower kept index in the low two bits;
//   B  dense column k of output column c sits in lane 16 ((k / 8) % 4) + c,
//      element (k % 8) + 8 (k / 32);
//   D  row r, column c in lane 16 (r / 4) + c, element r % 4.
// The export's metadata word holds the nibbles of 8 consecutive groups, group
// q at bits 4 (q % 8): a lane's 16 index bits are one half of one word.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kWaves = 4;

// One wave per 16 x 16 tile of Y [rows, tokens]; rows % 16 == 0,
// cols % 64 == 0, tokens % 16 == 0 (checked by the host).
__global__ __launch_bounds__(64 * kWaves) void sparse_mm_kernel(
    const uint16_t* vals, const uint32_t* meta, const uint16_t* X, float* Y, int64_t rows,
    int64_t cols, int64_t tokens)
{
    const int lane = threadIdx.x & 63;
    const int64_t tile = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
    const int64_t tiles_c = tokens / 16;
    if (tile >= (rows / 16) * tiles_c) return; // uniform over the wave
    const int64_t r0 = (tile / tiles_c) * 16, c0 = (tile % tiles_c) * 16;
    const int quad = lane >> 4;
    const int64_t r = r0 + (lane & 15);  // A row of this lane
    const int64_t c = c0 + (lane & 15);  // B column (token) of this lane
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int64_t k0 = 0; k0 < cols; k0 += 64) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(vals + r * (cols / 2) + k0 / 2 + 8 * quad);
        const uint32_t word = meta[(r * cols + k0) / 32 + quad / 2];
        const int idx = (int)((word >> (16 * (quad & 1))) & 0xFFFFu);
        const uint16_t* xr = X + c * cols + k0 + 8 * quad;
        const bf16x8 lo = *reinterpret_cast<const bf16x8*>(xr);
        const bf16x8 hi = *reinterpret_cast<const bf16x8*>(xr + 32);
        const bf16x16 b = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11,
                                                  12, 13, 14, 15);
        acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a, b, acc, idx, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) Y[(r0 + 4 * quad + i) * tokens + c0 + (lane & 15)] = acc[i];
}

} // namespace

// Y [rows, tokens] fp32 = W_sparse [rows, cols] (vals [rows, cols / 2] bf16,
// meta [rows * cols / 32] words) times X [tokens, cols] bf16, transposed.
// Returns 0, or -1 on a shape the kernel does not take, or the HIP error.
extern "C" int sparse_check_matmul_2of4(const uint16_t* vals, const uint32_t* meta,
                                        const uint16_t* X, float* Y, int64_t rows, int64_t cols,
                                        int64_t tokens, hipStream_t stream)
{
    if (!vals || !meta || !X || !Y || rows <= 0 || cols <= 0 || tokens <= 0 || rows % 16 ||
        cols % 64 || tokens % 16)
        return -1;
    const int64_t tiles = (rows / 16) * (tokens / 16);
    const int64_t blocks = (tiles + kWaves - 1) / kWaves;
    if (blocks > 0x7FFFFFFF) return -1;
    hipLaunchKernelGGL(sparse_mm_kernel, dim3((unsigned)blocks), dim3(64 * kWaves), 0, stream,
                       vals, meta, X, Y, rows, cols, tokens);
    return (int)hipGetLastError();
}
