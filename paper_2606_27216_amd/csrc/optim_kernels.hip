// Element-wise halves of the HiMuon optimizer step (Alg. 1) for the
// fused-kernel tile sizes, where the tile kernels themselves read and write
// plain matrices: a prologue that updates the momentum and forms the
// lookahead gradient into a contiguous buffer, and an epilogue that applies
// decoupled weight decay and the tau-scaled direction (eq. scaled_update)
// from that buffer. Memory-bound: each thread moves 8 consecutive elements
// of a row, with 16-byte accesses where the row chunk is whole and aligned.
#include "optim_kernels.h"
#include "elementwise8.h"

namespace himuon {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxGridY = 65535;  // one grid row per matrix

// Row chunk `ch` of matrix D: row r, columns c0 .. c0 + n - 1 (n <= 8).
struct Chunk {
    int64_t r, c0;
    int n;
};

__device__ __forceinline__ Chunk chunk_of(const StepDesc& D, int64_t ch)
{
    const int64_t cpr = (D.cols + 7) / 8;
    Chunk k;
    k.r = ch / cpr;
    k.c0 = (ch - k.r * cpr) * 8;
    k.n = (int)min<int64_t>(8, D.cols - k.c0);
    return k;
}

// M <- beta M + G (stored); buf <- G + beta M (Nesterov) or M.
template <GemmStore ST>
__global__ void __launch_bounds__(kThreads) step_lookahead(const StepDesc* descs, OptArgs o)
{
    const StepDesc D = descs[blockIdx.y];
    const int64_t n_ch = D.rows * ((D.cols + 7) / 8);
    for (int64_t ch = (int64_t)blockIdx.x * kThreads + threadIdx.x; ch < n_ch; ch += (int64_t)gridDim.x * kThreads) {
        const Chunk k = chunk_of(D, ch);
        const bool vec = D.vec && k.n == 8;
        const int64_t i = k.r * D.ld + k.c0;
        float g[8], m[8];
        load8<ST>(D.g, i, k.n, vec, g);
        load8<ST>(D.m, i, k.n, vec, m);
#pragma unroll
        for (int e = 0; e < 8; ++e) m[e] = o.beta * m[e] + g[e];
        store8<ST>(D.m, i, k.n, vec, m);
#pragma unroll
        for (int e = 0; e < 8; ++e) g[e] = o.nesterov ? g[e] + o.beta * m[e] : m[e];
        store8<ST>(D.buf, k.r * D.cols + k.c0, k.n, vec && D.vec_buf, g);
    }
}

// W <- (1 - lr lambda) W - lr tau U, U in buf.
template <GemmStore ST>
__global__ void __launch_bounds__(kThreads) step_apply(const StepDesc* descs, OptArgs o)
{
    const StepDesc D = descs[blockIdx.y];
    const int64_t n_ch = D.rows * ((D.cols + 7) / 8);
    const float step = o.lr * D.tau;
    for (int64_t ch = (int64_t)blockIdx.x * kThreads + threadIdx.x; ch < n_ch; ch += (int64_t)gridDim.x * kThreads) {
        const Chunk k = chunk_of(D, ch);
        const bool vec = D.vec && k.n == 8;
        const int64_t i = k.r * D.ld + k.c0;
        float w[8], u[8];
        load8<ST>(D.w, i, k.n, vec, w);
        load8<ST>(D.buf, k.r * D.cols + k.c0, k.n, vec && D.vec_buf, u);
#pragma unroll
        for (int e = 0; e < 8; ++e) w[e] = o.decay * w[e] - step * u[e];
        store8<ST>(D.w, i, k.n, vec, w);
    }
}

dim3 step_grid(int64_t max_chunks, int n_mats)
{
    const int64_t blocks = (max_chunks + kThreads - 1) / kThreads;
    return dim3((unsigned)std::min<int64_t>(std::max<int64_t>(blocks, 1), 4096), (unsigned)n_mats, 1);
}

}  // namespace

hipError_t launch_step_lookahead(GemmStore st, const StepDesc* descs, int n_mats, int64_t max_chunks,
                                 const OptArgs& o, hipStream_t stream)
{
    for (int l0 = 0; l0 < n_mats; l0 += kMaxGridY) {
        const dim3 grid = step_grid(max_chunks, std::min(kMaxGridY, n_mats - l0));
        if (st == GemmStore::BF16)
            hipLaunchKernelGGL(step_lookahead<GemmStore::BF16>, grid, dim3(kThreads), 0, stream, descs + l0, o);
        else
            hipLaunchKernelGGL(step_lookahead<GemmStore::F32>, grid, dim3(kThreads), 0, stream, descs + l0, o);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_step_apply(GemmStore st, const StepDesc* descs, int n_mats, int64_t max_chunks, const OptArgs& o,
                             hipStream_t stream)
{
    for (int l0 = 0; l0 < n_mats; l0 += kMaxGridY) {
        const dim3 grid = step_grid(max_chunks, std::min(kMaxGridY, n_mats - l0));
        if (st == GemmStore::BF16)
            hipLaunchKernelGGL(step_apply<GemmStore::BF16>, grid, dim3(kThreads), 0, stream, descs + l0, o);
        else
            hipLaunchKernelGGL(step_apply<GemmStore::F32>, grid, dim3(kThreads), 0, stream, descs + l0, o);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace himuon
