// Internal contract between the host planner (himuon_api.cpp) and the
// gfx950 kernel family (ns_tiled_kernels.hip). Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace himuon {

// One entry per matrix in a call; the table lives in the caller's workspace.
// Global tile ids are dense: matrix m owns [tile_begin, tile_begin + R*C),
// numbered row-major over its R x C tile grid.
struct alignas(64) MatDesc {
    const void* in;
    void* out;
    int64_t rows, cols;
    int64_t ld_in, ld_out;
    int64_t tile_begin;
    int32_t tiles_c;  // C = ceil(cols / T)
    int32_t flags;    // MAT_VEC_IN / MAT_VEC_OUT
};
static_assert(sizeof(MatDesc) == 64, "descriptor layout");

// Base pointer and leading dimension allow 16-byte accesses at every column
// that is a multiple of 8 (bf16) or 4 (f32).
constexpr int32_t MAT_VEC_IN = 1;
constexpr int32_t MAT_VEC_OUT = 2;

enum class Storage : int { F32 = 0, BF16 = 1 };
enum class Operand : int { F32 = 1, F16 = 2, BF16 = 3 };

// Kernel arguments of one chunk launch: tiles [tile_begin, tile_end).
struct KernelArgs {
    const MatDesc* descs;
    int64_t tile_begin;
    int64_t tile_end;
    int32_t n_mats;
    int32_t K;
    float a, b, c;
    float b_over_c;  // b / c, used when c != 0
    // Rescaled state Z = X |c|^(1/4) (fp16-operand kernel; c != 0):
    // Z <- aZ + sigma H (H + sigma b' I) Z with H = Z Z^T, b' = b / sqrt|c|.
    float zscale;    // |c|^(1/4) (1 when c == 0)
    float unscale;   // 1 / zscale
    float bq;        // sigma * b' (c != 0) or b (c == 0)
    float sigma;     // sign(c), 0 when c == 0
};

// Enqueue one chunk on `stream`. Returns hipErrorInvalidValue for a
// (T, storage, operand) triple without a kernel.
hipError_t launch_ns_tiled(int T, Storage st, Operand op, const KernelArgs& args, hipStream_t stream);

// True when a kernel exists for the triple (no HIP call).
bool has_kernel(int T, Storage st, Operand op);

// The fp16-operand kernel family (bf16 storage), T in {32, 64, 128, 256}.
hipError_t launch_ns_tiled_f16(int T, const KernelArgs& args, hipStream_t stream);

// Host helpers shared by the entry points (himuon_api.cpp).
extern thread_local int g_last_hip_error;
// Records `e` as the calling thread's last HIP error; returns HIMUON_ERR_HIP.
int set_hip_error(hipError_t e);
// Copies `bytes` of host data to device memory `dst` on `stream` through a
// ring of pinned staging slots (asynchronous; a slot is reused once its
// copy has completed). Returns a himuon status.
int upload_table(const void* data, size_t bytes, void* dst, hipStream_t stream, int dev);
// Largest |p^k(s)| over s in [0, 1], k < K, p(s) = a s + b s^3 + c s^5.
double iterate_bound(int K, double a, double b, double c);

}  // namespace himuon
