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
    float tau;           // optimizer step: the update scale tau of the block's matrix
    void* mom;           // optimizer step: the momentum buffer (layout of `in`)
    int32_t vec;         // GEMM_VEC_IN / GEMM_VEC_OUT
    int32_t pad0_;
    int64_t pad_[6];
};
static_assert(sizeof(GemmProb) == 128, "problem descriptor layout");

// Every 8-column chunk of the block's rows that starts at a multiple of 8
// is 16-byte aligned in `in` and `mom` (GEMM_VEC_IN) or in `out` (GEMM_VEC_OUT).
constexpr int32_t GEMM_VEC_IN = 1;
constexpr int32_t GEMM_VEC_OUT = 2;

// The optimizer step of Alg. 1 fused into the gather and scatter kernels:
// `in` holds the gradient G, `mom` the momentum M and `out` the weights W.
// The gather stores M <- beta M + G (rounded to the storage type) and takes
// the problem's input as G + beta M (Nesterov) or M; the scatter stores
// W <- (1 - lr lambda) W - lr tau U, eq. (scaled_update).
struct OptArgs {
    float beta;
    float decay;  // 1 - lr * lambda
    float lr;
    int32_t nesterov;
};

// Element types: storage (what the caller's matrices hold) and the GEMM
// operand type of the iterate.
enum class GemmStore : int { F32 = 0, BF16 = 1 };
enum class GemmOperand : int { F32 = 1, F16 = 2, BF16 = 3 };

// Partial sums of squares, fp64: part j of problem p covers a fixed slice
// of its h x w block; result at partial[p * nparts + j].
hipError_t launch_gemm_norm_partials(GemmStore st, const GemmProb* probs, int nprob, int nparts,
                                     double* partial, const OptArgs* opt, hipStream_t stream);

// X0 = scale * B / ||B||_F (zero when the block is zero) as the m x n
// row-major iterate of each problem, stride m * n elements.
hipError_t launch_gemm_gather(GemmStore st, GemmOperand op, const GemmProb* probs, int nprob, int m, int n,
                              int nparts, const double* partial, double scale, void* x, const OptArgs* opt,
                              hipStream_t stream);

// Output block = inv_scale * (the block's part of the iterate), rounded to
// the storage type (nearest even for bf16).
hipError_t launch_gemm_scatter(GemmStore st, GemmOperand op, const GemmProb* probs, int nprob, int m, int n,
                               float inv_scale, const void* x, const OptArgs* opt, hipStream_t stream);

// Core of himuon_ns_gemm(_hw) and of the optimizer step on the GEMM path
// (`opt` null: Phi of `in` into `out`), with Th x Tw tiles (0 x 0: whole
// matrices). Returns a himuon status.
int run_gemm_path(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, void* const* mom_ptrs,
                  const float* tau, const int64_t* rows, const int64_t* cols, const int64_t* ld_in,
                  const int64_t* ld_out, int Th, int Tw, int K, float a, float b, float c, int dtype, int compute,
                  void* workspace, size_t workspace_bytes, size_t chunk_budget_bytes, void* stream,
                  const OptArgs* opt);
// Workspace of run_gemm_path (0 when the call has no plan).
size_t gemm_path_workspace(int64_t n_mats, const int64_t* rows, const int64_t* cols, int Th, int Tw, int dtype,
                           int compute, int K, float a, float b, float c, size_t chunk_budget_bytes);

}  // namespace himuon
