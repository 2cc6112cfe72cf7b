// Eight consecutive elements of a row as fp32, for the memory-bound kernels
// (gather/scatter of the library-GEMM path and the optimizer-step
// prologue/epilogue). `vec` selects one 16-byte access (bf16) or two (fp32);
// it requires the chunk to be whole (n == 8) and 16-byte aligned. Elements
// at or beyond n read as zero and are not written.
#pragma once

#include "ns_gemm_path.h"

#include <hip/hip_bf16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace himuon {

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

}  // namespace himuon
