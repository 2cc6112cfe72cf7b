// Gather, normalisation and scatter kernels of the library-GEMM path
// (whole matrices and large tiles). The Newton-Schulz steps themselves are
// three library GEMMs per step (see ns_gemm_path.cpp); these kernels move a
// problem's block between the caller's matrix and the iterate buffer:
//   - B_T (Sec. 2.1, eq. tiling_operator): the block at the top left of an
//     m x n iterate, zero elsewhere; a whole matrix with more rows than
//     columns is taken transposed (Phi_K(S^T) = Phi_K(S)^T), so the Gram
//     matrix is the smaller one;
//   - the normalisation X0 = S / ||S||_F of Phi_K (Sec. 2.2, eq. phi_k_def;
//     Phi_K(0) = 0), with the norm summed in fp64 in a fixed order, so a
//     result never depends on how problems are grouped into launches;
//   - B_T^{-1}: the block part of the final iterate back to the matrix.
// With the optimizer step of Alg. 1 fused in (OPT), the problem's input is
// the lookahead gradient formed on the fly from G and the momentum M (the
// norm pass also stores the new M), and the scatter applies the decoupled
// weight decay and the tau-scaled update to W (eq. scaled_update).
#include "ns_gemm_path.h"
#include "elementwise8.h"

#include <hip/hip_bf16.h>
#include <hip/hip_fp16.h>
#include <math.h>

namespace himuon {
namespace {

constexpr int kThreads = 256;
// A block of the gather and scatter covers 32 rows x 64 columns of the
// iterate: in the row-major orientation a thread moves one 8-column chunk;
// a transposed block goes through LDS as two 32 x 32 tiles, four rows per
// thread.
constexpr int kBlkRows = 32, kBlkCols = 64;

template <GemmStore ST>
__device__ __forceinline__ void store_elem(void* base, int64_t idx, float v)
{
    if constexpr (ST == GemmStore::BF16) {
        const __bf16 h = (__bf16)v;  // round to nearest even
        static_cast<__bf16*>(base)[idx] = h;
    } else {
        static_cast<float*>(base)[idx] = v;
    }
}

template <GemmStore ST>
__device__ __forceinline__ float load_f32(const void* base, int64_t idx)
{
    if constexpr (ST == GemmStore::BF16) {
        const uint16_t u = static_cast<const uint16_t*>(base)[idx];
        return __uint_as_float((uint32_t)u << 16);
    } else {
        return static_cast<const float*>(base)[idx];
    }
}

// Eq. (muon_lookahead) or the plain buffer, from G and the stored new M.
__device__ __forceinline__ float lookahead(float g, float m_new, const OptArgs& o)
{
    return o.nesterov ? g + o.beta * m_new : m_new;
}

// Element `idx` of the problem's input: the matrix itself, or (OPT) the
// lookahead gradient from G (`in`) and the already updated momentum.
template <GemmStore ST, bool OPT>
__device__ __forceinline__ float input_elem(const GemmProb& P, int64_t idx, const OptArgs& o)
{
    if constexpr (OPT) return lookahead(load_f32<ST>(P.in, idx), load_f32<ST>(P.mom, idx), o);
    else return load_f32<ST>(P.in, idx);
}

// Writes the result u of element `idx`: the plain output, or (OPT) the
// weight update W <- (1 - lr lambda) W - lr tau u.
template <GemmStore ST, bool OPT>
__device__ __forceinline__ void output_elem(const GemmProb& P, int64_t idx, float u, const OptArgs& o)
{
    if constexpr (OPT) {
        const float w = load_f32<ST>(P.out, idx);
        store_elem<ST>(P.out, idx, o.decay * w - (o.lr * P.tau) * u);
    } else {
        store_elem<ST>(P.out, idx, u);
    }
}

template <GemmOperand OP> struct OpType;
template <> struct OpType<GemmOperand::F32> { typedef float T; };
template <> struct OpType<GemmOperand::F16> { typedef _Float16 T; };
template <> struct OpType<GemmOperand::BF16> { typedef __bf16 T; };

// Part j of problem p sums the squares of rows [j*rpp, (j+1)*rpp) of its
// block, each thread over a fixed set of columns, then a fixed-order tree.
// (OPT: the momentum update M <- beta M + G of every element happens here,
// once, and the sum is over the lookahead gradient formed from its stored
// value, exactly as the gather forms it.)
template <GemmStore ST, bool OPT>
__global__ void __launch_bounds__(kThreads) gemm_norm_partials(const GemmProb* probs, int nparts, double* partial,
                                                               const OptArgs o)
{
    const GemmProb P = probs[blockIdx.y];
    const int rpp = (P.h + nparts - 1) / nparts;
    const int r0 = (int)blockIdx.x * rpp;
    const int r1 = min(P.h, r0 + rpp);
    double acc = 0.0;
    // the part's rows x 8-column chunks, flattened: element e = (row, chunk)
    const int cpr = (P.w + 7) / 8;
    const int64_t n_e = (int64_t)max(r1 - r0, 0) * cpr;
    for (int64_t e0 = threadIdx.x; e0 < n_e; e0 += kThreads) {
        const int r = r0 + (int)(e0 / cpr), c = 8 * (int)(e0 % cpr);
        const int64_t rowoff = (P.row0 + r) * P.ld_in + P.col0;
        const int nv = min(8, P.w - c);
        const bool vec = (P.vec & GEMM_VEC_IN) && nv == 8;
        float g[8];
        load8<ST>(P.in, rowoff + c, nv, vec, g);
        if constexpr (OPT) {
            float m[8];
            load8<ST>(P.mom, rowoff + c, nv, vec, m);
#pragma unroll
            for (int e = 0; e < 8; ++e) m[e] = o.beta * m[e] + g[e];
            store8<ST>(P.mom, rowoff + c, nv, vec, m);
#pragma unroll
            for (int e = 0; e < 8; ++e) g[e] = lookahead(g[e], m[e], o);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) acc += (double)g[e] * (double)g[e];
    }
    __shared__ double red[kThreads];
    red[threadIdx.x] = acc;
    __syncthreads();
#pragma unroll
    for (int s = kThreads / 2; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) partial[(int64_t)blockIdx.y * nparts + blockIdx.x] = red[0];
}

// The problem's scale factor, scale / ||B||_F (0 for a zero block), written
// over its first partial.
__global__ void gemm_norm_finalize(int nprob, int nparts, double scale, double* partial)
{
    const int p = blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= nprob) return;
    double ss = 0.0;
    for (int j = 0; j < nparts; ++j) ss += partial[(int64_t)p * nparts + j];
    partial[(int64_t)p * nparts] = ss > 0.0 ? scale / sqrt(ss) : 0.0;
}

// Eight consecutive iterate elements (operand type) as fp32 / from fp32;
// `vec` when the chunk is whole and 16-byte aligned.
template <GemmOperand OP>
__device__ __forceinline__ void load_x8(const void* xv, int64_t idx, int n, bool vec, float (&v)[8])
{
    typedef typename OpType<OP>::T OT;
    const OT* x = static_cast<const OT*>(xv) + idx;
    if constexpr (OP == GemmOperand::F32) {
        load8<GemmStore::F32>(x, 0, n, vec, v);
    } else {
        if (vec) {
            const uint4 r = *reinterpret_cast<const uint4*>(x);
            const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint16_t h = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
                v[e] = (float)__builtin_bit_cast(OT, h);
            }
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = e < n ? (float)x[e] : 0.f;
        }
    }
}

template <GemmOperand OP>
__device__ __forceinline__ void store_x8(void* xv, int64_t idx, int n, bool vec, const float (&v)[8])
{
    typedef typename OpType<OP>::T OT;
    OT* x = static_cast<OT*>(xv) + idx;
    if constexpr (OP == GemmOperand::F32) {
        float t[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) t[e] = v[e];
        store8<GemmStore::F32>(x, 0, n, vec, t);
    } else {
        if (vec) {
            uint16_t h[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) h[e] = __builtin_bit_cast(uint16_t, (OT)v[e]);
            uint4 r;
            r.x = h[0] | ((uint32_t)h[1] << 16);
            r.y = h[2] | ((uint32_t)h[3] << 16);
            r.z = h[4] | ((uint32_t)h[5] << 16);
            r.w = h[6] | ((uint32_t)h[7] << 16);
            *reinterpret_cast<uint4*>(x) = r;
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (e < n) x[e] = (OT)v[e];
        }
    }
}

template <GemmStore ST, GemmOperand OP, bool OPT>
__global__ void __launch_bounds__(kThreads) gemm_gather(const GemmProb* probs, int m, int n, int nparts,
                                                        const double* partial, void* xv, const OptArgs o)
{
    typedef typename OpType<OP>::T OT;
    const int p = blockIdx.y;
    const GemmProb P = probs[p];
    const double s = partial[(int64_t)p * nparts];
    const int blk_n = (n + kBlkCols - 1) / kBlkCols;
    const int i0 = (int)(blockIdx.x / blk_n) * kBlkRows, j0 = (int)(blockIdx.x % blk_n) * kBlkCols;
    OT* x = static_cast<OT*>(xv) + (int64_t)p * m * n;
    if (!P.trans) {
        const int i = i0 + (int)(threadIdx.x >> 3), j = j0 + 8 * (int)(threadIdx.x & 7);
        if (i >= m || j >= n) return;
        float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        if (i < P.h && j < P.w) {
            const int nv = min(8, P.w - j);
            const bool vec = (P.vec & GEMM_VEC_IN) && nv == 8;
            const int64_t idx = (P.row0 + i) * P.ld_in + P.col0 + j;
            load8<ST>(P.in, idx, nv, vec, v);
            if constexpr (OPT) {
                float mm[8];
                load8<ST>(P.mom, idx, nv, vec, mm);
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = lookahead(v[e], mm[e], o);
            }
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (float)((double)v[e] * s);
        store_x8<OP>(x, (int64_t)i * n + j, min(8, n - j), n % 8 == 0, v);
    } else {
        // iterate (i, j) = block (j, i): block rows j0.., columns i0.. through LDS
        __shared__ float t[32][33];
        const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
        for (int half = 0; half < 2; ++half) {
            const int jh = j0 + 32 * half;
            if (half) __syncthreads();
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int r = jh + ty + 8 * k, c = i0 + tx;
                double v = 0.0;
                if (r < P.h && c < P.w) v = (double)input_elem<ST, OPT>(P, (P.row0 + r) * P.ld_in + P.col0 + c, o) * s;
                t[ty + 8 * k][tx] = (float)v;
            }
            __syncthreads();
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int i = i0 + ty + 8 * k, j = jh + tx;
                if (i < m && j < n) x[(int64_t)i * n + j] = (OT)t[tx][ty + 8 * k];
            }
        }
    }
}

template <GemmStore ST, GemmOperand OP, bool OPT>
__global__ void __launch_bounds__(kThreads) gemm_scatter(const GemmProb* probs, int m, int n, float inv_scale,
                                                         const void* xv, const OptArgs o)
{
    typedef typename OpType<OP>::T OT;
    const int p = blockIdx.y;
    const GemmProb P = probs[p];
    const int blk_n = (n + kBlkCols - 1) / kBlkCols;
    const int i0 = (int)(blockIdx.x / blk_n) * kBlkRows, j0 = (int)(blockIdx.x % blk_n) * kBlkCols;
    const OT* x = static_cast<const OT*>(xv) + (int64_t)p * m * n;
    if (!P.trans) {
        const int i = i0 + (int)(threadIdx.x >> 3), j = j0 + 8 * (int)(threadIdx.x & 7);
        if (i >= P.h || j >= P.w) return;
        const int nv = min(8, P.w - j);
        float u[8];
        load_x8<OP>(x, (int64_t)i * n + j, nv, n % 8 == 0 && nv == 8, u);
#pragma unroll
        for (int e = 0; e < 8; ++e) u[e] *= inv_scale;
        const bool vec = (P.vec & GEMM_VEC_OUT) && nv == 8;
        const int64_t idx = (P.row0 + i) * P.ld_out + P.col0 + j;
        if constexpr (OPT) {
            float w[8];
            load8<ST>(P.out, idx, nv, vec, w);
            const float step = o.lr * P.tau;
#pragma unroll
            for (int e = 0; e < 8; ++e) w[e] = o.decay * w[e] - step * u[e];
            store8<ST>(P.out, idx, nv, vec, w);
        } else {
            store8<ST>(P.out, idx, nv, vec, u);
        }
    } else {
        __shared__ float t[32][33];
        const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
        for (int half = 0; half < 2; ++half) {
            const int jh = j0 + 32 * half;
            if (half) __syncthreads();
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int i = i0 + ty + 8 * k, j = jh + tx;
                t[ty + 8 * k][tx] = (i < m && j < n) ? (float)x[(int64_t)i * n + j] * inv_scale : 0.f;
            }
            __syncthreads();
            // block (r, c) = iterate (c, r): block rows jh.., columns i0..
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int r = jh + ty + 8 * k, c = i0 + tx;
                if (r < P.h && c < P.w) output_elem<ST, OPT>(P, (P.row0 + r) * P.ld_out + P.col0 + c, t[tx][ty + 8 * k], o);
            }
        }
    }
}

dim3 tile_grid(int m, int n, int nprob)
{
    return dim3((unsigned)(((m + kBlkRows - 1) / kBlkRows) * ((n + kBlkCols - 1) / kBlkCols)), (unsigned)nprob, 1);
}

}  // namespace

hipError_t launch_gemm_norm_partials(GemmStore st, const GemmProb* probs, int nprob, int nparts, double* partial,
                                     const OptArgs* opt, hipStream_t stream)
{
    if (nprob <= 0) return hipSuccess;
    const dim3 grid((unsigned)nparts, (unsigned)nprob, 1);
    const OptArgs o = opt ? *opt : OptArgs{};
#define HM_NORM(S, F) \
    hipLaunchKernelGGL((gemm_norm_partials<S, F>), grid, dim3(kThreads), 0, stream, probs, nparts, partial, o)
    if (st == GemmStore::BF16) {
        if (opt) HM_NORM(GemmStore::BF16, true);
        else HM_NORM(GemmStore::BF16, false);
    } else {
        if (opt) HM_NORM(GemmStore::F32, true);
        else HM_NORM(GemmStore::F32, false);
    }
#undef HM_NORM
    return hipGetLastError();
}

hipError_t launch_gemm_gather(GemmStore st, GemmOperand op, const GemmProb* probs, int nprob, int m, int n,
                              int nparts, const double* partial, double scale, void* x, const OptArgs* opt,
                              hipStream_t stream)
{
    if (nprob <= 0) return hipSuccess;
    hipLaunchKernelGGL(gemm_norm_finalize, dim3((unsigned)((nprob + 255) / 256)), dim3(256), 0, stream, nprob, nparts,
                       scale, const_cast<double*>(partial));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid = tile_grid(m, n, nprob);
    const OptArgs o = opt ? *opt : OptArgs{};
#define HM_GATHER(S, O)                                                                                              \
    do {                                                                                                             \
        if (opt)                                                                                                     \
            hipLaunchKernelGGL((gemm_gather<S, O, true>), grid, dim3(kThreads), 0, stream, probs, m, n, nparts,      \
                               partial, x, o);                                                                       \
        else                                                                                                         \
            hipLaunchKernelGGL((gemm_gather<S, O, false>), grid, dim3(kThreads), 0, stream, probs, m, n, nparts,     \
                               partial, x, o);                                                                       \
    } while (0)
    if (st == GemmStore::F32 && op == GemmOperand::F32) HM_GATHER(GemmStore::F32, GemmOperand::F32);
    else if (st == GemmStore::BF16 && op == GemmOperand::F16) HM_GATHER(GemmStore::BF16, GemmOperand::F16);
    else if (st == GemmStore::BF16 && op == GemmOperand::BF16) HM_GATHER(GemmStore::BF16, GemmOperand::BF16);
    else return hipErrorInvalidValue;
#undef HM_GATHER
    return hipGetLastError();
}

hipError_t launch_gemm_scatter(GemmStore st, GemmOperand op, const GemmProb* probs, int nprob, int m, int n,
                               float inv_scale, const void* x, const OptArgs* opt, hipStream_t stream)
{
    if (nprob <= 0) return hipSuccess;
    const dim3 grid = tile_grid(m, n, nprob);
    const OptArgs o = opt ? *opt : OptArgs{};
#define HM_SCATTER(S, O)                                                                                             \
    do {                                                                                                             \
        if (opt)                                                                                                     \
            hipLaunchKernelGGL((gemm_scatter<S, O, true>), grid, dim3(kThreads), 0, stream, probs, m, n, inv_scale,  \
                               x, o);                                                                                \
        else                                                                                                         \
            hipLaunchKernelGGL((gemm_scatter<S, O, false>), grid, dim3(kThreads), 0, stream, probs, m, n, inv_scale, \
                               x, o);                                                                                \
    } while (0)
    if (st == GemmStore::F32 && op == GemmOperand::F32) HM_SCATTER(GemmStore::F32, GemmOperand::F32);
    else if (st == GemmStore::BF16 && op == GemmOperand::F16) HM_SCATTER(GemmStore::BF16, GemmOperand::F16);
    else if (st == GemmStore::BF16 && op == GemmOperand::BF16) HM_SCATTER(GemmStore::BF16, GemmOperand::BF16);
    else return hipErrorInvalidValue;
#undef HM_SCATTER
    return hipGetLastError();
}

}  // namespace himuon
