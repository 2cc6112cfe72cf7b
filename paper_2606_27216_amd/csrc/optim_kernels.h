// Internal contract of the element-wise optimizer-step kernels used with
// the fused tile kernels (T in {32, 64, 128, 256}). Not part of the public ABI.
#pragma once

#include "ns_gemm_path.h"

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace himuon {

// One matrix of the step: weights w, gradient g and momentum m share the
// row-major layout (leading dimension ld); buf is a contiguous rows x cols
// buffer that receives the lookahead gradient and, after the tiled map ran
// on it in place, holds the direction U.
struct alignas(64) StepDesc {
    void* w;
    const void* g;
    void* m;
    void* buf;
    int64_t rows, cols, ld;
    float tau;
    uint16_t vec;      // w, g, m allow 16-byte accesses at every 8th column
    uint16_t vec_buf;  // buf does
};
static_assert(sizeof(StepDesc) == 64, "step descriptor layout");

// M <- beta M + G (rounded to storage), buf <- G + beta M or M (Alg. 1).
// `max_chunks`: the largest rows * ceil(cols / 8) over the matrices.
hipError_t launch_step_lookahead(GemmStore st, const StepDesc* descs, int n_mats, int64_t max_chunks,
                                 const OptArgs& o, hipStream_t stream);
// W <- (1 - lr lambda) W - lr tau buf (eq. scaled_update).
hipError_t launch_step_apply(GemmStore st, const StepDesc* descs, int n_mats, int64_t max_chunks, const OptArgs& o,
                             hipStream_t stream);

}  // namespace himuon
