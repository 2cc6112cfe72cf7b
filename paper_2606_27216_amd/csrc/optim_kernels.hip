// Element-wise halves of the HiMuon optimizer step (Alg. 1) for the
// fused-kernel tile sizes, where the tile kernels themselves read and write
// plain matrices: a prologue that updates the momentum and forms the
// lookahead gradient into a contiguous buffer, and an epilogue that applies
// decoupled weight decay and the tau-scaled direction (eq. scaled_update)
// from that buffer. Memory-bound: each thread moves 8 consecutive elements
// of a row, with 16-byte accesses where the row chunk is whole and aligned.
#include "optim_kernels.h"

#include <hip/hip_bf16.h>

namespace himuon {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxGridY = 65535;  // one grid row per matrix

template <GemmStore ST>
__device__ __forceinline__ void load8(const void* base, int64_t idx, int n, bool vec, float (&v)[8])
{
    if constexpr (ST == GemmStore::BF16) {
        const uint16_t* p = static_cast<const uint16_t*>(base) + idx;
        if (vec) {
            const uint4 r = *reinterpret_cast<const uint4*>(p);
            const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = __uint_as_float((e & 1) ? (w[e >> 1] & 0xffff0000u) : (w[e >> 1] << 16));
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = e < n ? __uint_as_float((uint32_t)p[e] << 16) : 0.f;
        }
    } else {
        const float* p = static_cast<const float*>(base) + idx;
        if (vec) {
            const float4 a = *reinterpret_cast<const float4*>(p);
            const float4 b = *reinterpret_cast<const float4*>(p + 4);
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
            v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = e < n ? p[e] : 0.f;
        }
    }
}

// Stores v rounded to the storage type (nearest even for bf16) and leaves
// the stored values in v.
template <GemmStore ST>
__device__ __forceinline__ void store8(void* base, int64_t idx, int n, bool vec, float (&v)[8])
{
    if constexpr (ST == GemmStore::BF16) {
        uint16_t h[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const __bf16 b = (__bf16)v[e];
            h[e] = __builtin_bit_cast(uint16_t, b);
            v[e] = (float)b;
        }
        uint16_t* p = static_cast<uint16_t*>(base) + idx;
        if (vec) {
            uint4 r;
            r.x = h[0] | ((uint32_t)h[1] << 16);
            r.y = h[2] | ((uint32_t)h[3] << 16);
            r.z = h[4] | ((uint32_t)h[5] << 16);
            r.w = h[6] | ((uint32_t)h[7] << 16);
            *reinterpret_cast<uint4*>(p) = r;
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (e < n) p[e] = h[e];
        }
    } else {
        float* p = static_cast<float*>(base) + idx;
        if (vec) {
            *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
            *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (e < n) p[e] = v[e];
        }
    }
}

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
