// Measurement aid, not part of the map: the MFMA rate this device sustains
// when it runs nothing but dense 32x32x16 products, the ceiling against which
// the tile kernels' issued MFMA work is read (their products are the same
// instructions, with operands, conversions and memory traffic around them).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "himuon.h"
#include "himuon_internal.h"

namespace himuon {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCalibThreads = 256;
constexpr int kCalibOperands = 4096;  // 16-byte operand words read from `ops`
constexpr int kCalibMaxGrid = 1 << 20;  // keeps 4 * (global lane index) within int

// Every wave keeps four independent accumulators (so no product waits on
// the one before it) and issues 4 * iters products on operands loaded once;
// the sums land in `out` so that nothing is optimised away.
template <bool BF16>
__global__ void __launch_bounds__(kCalibThreads) calib_mfma_kernel(const u32x4* ops, float* out, int iters)
{
    const int l = threadIdx.x + blockIdx.x * kCalibThreads;
    const u32x4 a0 = ops[(4 * l + 0) % kCalibOperands], a1 = ops[(4 * l + 1) % kCalibOperands];
    const u32x4 b0 = ops[(4 * l + 2) % kCalibOperands], b1 = ops[(4 * l + 3) % kCalibOperands];
    f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int i = 0; i < iters; ++i) {
        if constexpr (BF16) {
            const bf16x8 x0 = __builtin_bit_cast(bf16x8, a0), x1 = __builtin_bit_cast(bf16x8, a1);
            const bf16x8 y0 = __builtin_bit_cast(bf16x8, b0), y1 = __builtin_bit_cast(bf16x8, b1);
            c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x0, y0, c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x1, y0, c1, 0, 0, 0);
            c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x0, y1, c2, 0, 0, 0);
            c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x1, y1, c3, 0, 0, 0);
        } else {
            const f16x8 x0 = __builtin_bit_cast(f16x8, a0), x1 = __builtin_bit_cast(f16x8, a1);
            const f16x8 y0 = __builtin_bit_cast(f16x8, b0), y1 = __builtin_bit_cast(f16x8, b1);
            c0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(x0, y0, c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(x1, y0, c1, 0, 0, 0);
            c2 = __builtin_amdgcn_mfma_f32_32x32x16_f16(x0, y1, c2, 0, 0, 0);
            c3 = __builtin_amdgcn_mfma_f32_32x32x16_f16(x1, y1, c3, 0, 0, 0);
        }
    }
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) s += (c0[v] + c1[v]) + (c2[v] + c3[v]);
    out[l] = s;
}

}  // namespace
}  // namespace himuon

extern "C" int himuon_calib_mfma(int compute, const void* ops, float* out, int grid, int iters, void* stream)
{
    using namespace himuon;
    if (!ops || !out || grid < 1 || grid > kCalibMaxGrid || iters < 1) return HIMUON_ERR_INVALID_ARG;
    if (compute != HIMUON_COMPUTE_F16 && compute != HIMUON_COMPUTE_BF16) return HIMUON_ERR_INVALID_ARG;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    if (compute == HIMUON_COMPUTE_BF16)
        hipLaunchKernelGGL(calib_mfma_kernel<true>, dim3(grid), dim3(kCalibThreads), 0, hs, (const u32x4*)ops, out, iters);
    else
        hipLaunchKernelGGL(calib_mfma_kernel<false>, dim3(grid), dim3(kCalibThreads), 0, hs, (const u32x4*)ops, out, iters);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? HIMUON_OK : set_hip_error(e);
}
