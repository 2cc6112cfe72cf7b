// Internal contract of the library-GEMM path (whole matrices, T = 0, and
// large tiles such as T = 512): the per-problem descriptor the gather and
// scatter kernels read, and their launchers. Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace himuon {

// One Newton-Schulz problem: an h x w block of a matrix (a T x T tile, or
// the whole matrix) worked on as an m x n iterate with m <= n. The block
// sits at the top left of the iterate and the rest is zero (the padding of
// the tiling operator). With `trans` the iterate is the block's transpose
// (a whole matrix with more rows than columns), so that the Gram matrix is
// the smaller one.
struct alignas(64) GemmProb {
    const void* in;
    void* out;
    int64_t ld_in, ld_out;
    int64_t row0, col0;  // origin of the block in the matrix
    int32_t h, w;        // block rows, columns (in the matrix's orientation)
    int32_t trans;
    int32_t pad_;
};
static_assert(sizeof(GemmProb) == 64, "problem descriptor layout");

// Element types: storage (what the caller's matrices hold) and the GEMM
// operand type of the iterate.
enum class GemmStore : int { F32 = 0, BF16 = 1 };
enum class GemmOperand : int { F32 = 1, F16 = 2, BF16 = 3 };

// Partial sums of squares, fp64: part j of problem p covers a fixed slice
// of its h x w block; result at partial[p * nparts + j].
hipError_t launch_gemm_norm_partials(GemmStore st, const GemmProb* probs, int nprob, int nparts,
                                     double* partial, hipStream_t stream);

// X0 = scale * B / ||B||_F (zero when the block is zero) as the m x n
// row-major iterate of each problem, stride m * n elements.
hipError_t launch_gemm_gather(GemmStore st, GemmOperand op, const GemmProb* probs, int nprob, int m, int n,
                              int nparts, const double* partial, double scale, void* x, hipStream_t stream);

// Output block = inv_scale * (the block's part of the iterate), rounded to
// the storage type (nearest even for bf16).
hipError_t launch_gemm_scatter(GemmStore st, GemmOperand op, const GemmProb* probs, int nprob, int m, int n,
                               float inv_scale, const void* x, hipStream_t stream);

}  // namespace himuon
