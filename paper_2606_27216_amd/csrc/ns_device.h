// Device-side helpers shared by the tiled Newton–Schulz kernel sources:
// vector types, MFMA operand packing, lane exchanges, the constant-space
// view of the descriptor table and the tile gather/scatter primitives.
#pragma once

#include "himuon_internal.h"

#include <stddef.h>

#include <math.h>

namespace himuon {
namespace dev {


typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// 16-byte vectors in the global address space (global_load / global_store)
typedef __attribute__((address_space(1))) u32x4 gbl_u32x4;

#define HM_DEV __device__ __forceinline__

// The descriptor table is written before a launch and only read during it,
// so the kernels read it through the constant address space: uniform
// descriptor loads become scalar loads, which do not wait on the vector
// memory counter that the tile loads and stores share.
typedef __attribute__((address_space(4))) const MatDesc ConstDesc;
typedef __attribute__((address_space(4))) const OptDesc ConstOpt;
// A table carried in the arguments is read where the launch placed them:
// every kernel that reads these tables takes its KernelArgs as its first
// argument, at offset 0 of the kernel-argument segment. (Addressing the
// argument itself instead would make the compiler copy the whole structure
// into per-lane scratch memory.)
typedef __attribute__((address_space(4))) const uint8_t ConstByte;
HM_DEV ConstByte* kernarg_base() { return (ConstByte*)__builtin_amdgcn_kernarg_segment_ptr(); }
HM_DEV const ConstDesc* desc_table(const KernelArgs& a)
{
    if (a.descs) return (const ConstDesc*)(uintptr_t)a.descs;
    return (const ConstDesc*)(kernarg_base() + offsetof(KernelArgs, inline_descs));
}
HM_DEV const ConstOpt* opt_table(const KernelArgs& a)
{
    if (a.odescs) return (const ConstOpt*)(uintptr_t)a.odescs;
    return (const ConstOpt*)(kernarg_base() + offsetof(KernelArgs, inline_odescs));
}

// Matrix owning `tile`, searching from `hint` (the tiles one wave visits only
// grow, so the owner of an earlier tile is a lower bound). Tile ids of one
// call fit in 32 bits (the host rejects larger calls), so every comparison is
// a scalar 32-bit one. The first tiles of the next four matrices are loaded
// unconditionally (indices clamped to the table), so the four scalar loads go
// out together and the usual case costs one round trip; a binary search
// covers the rest.
HM_DEV int find_matrix_from(const KernelArgs& args, int64_t tile, int hint)
{
    const ConstDesc* const descs = desc_table(args);
    constexpr int kAhead = 4;
    const uint32_t t = (uint32_t)tile;
    uint32_t tb[kAhead];
#pragma unroll
    for (int j = 0; j < kAhead; ++j) tb[j] = (uint32_t)descs[min(hint + 1 + j, args.n_mats - 1)].tile_begin;
    int passed = 0;
#pragma unroll
    for (int j = 0; j < kAhead; ++j) passed += (hint + 1 + j < args.n_mats && tb[j] <= t) ? 1 : 0;
    if (passed < kAhead) return hint + passed;
    int lo = hint + kAhead, hi = args.n_mats - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((uint32_t)descs[mid].tile_begin <= t) lo = mid;
        else hi = mid - 1;
    }
    return __builtin_amdgcn_readfirstlane(lo);
}

// 16-byte operand slots per lane per 32x32 block: a slot feeds one
// 32x32x16 fp16/bf16 MFMA (8 values) or four 32x32x2 fp32 MFMAs (4 values).
// kChains: independent accumulators per output block. The fp32 path spreads
// the four k-pairs of a slot over four chains (summed at the end of each
// product), which shortens every fp32 rounding walk four-fold; 16-bit
// operands round far above that level and use one chain.
template <Operand OP> struct OperandTraits {
    static constexpr int kSlots = 2;
    static constexpr int kChains = 1;
};
template <> struct OperandTraits<Operand::F32> {
    static constexpr int kSlots = 4;
    static constexpr int kChains = 4;
};

typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 values rounded to nearest even and packed (v_cvt_pk_{f16,bf16}_f32).
template <Operand OP> HM_DEV uint32_t pack2(float x, float y)
{
    const f32x2 v = {x, y};
    if constexpr (OP == Operand::F16) return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2));
    else return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Slot s of a row piece: values 8s..8s+7 (16-bit) or 4s..4s+3 (fp32).
template <Operand OP> HM_DEV u32x4 make_slot(const f32x16& v, int s)
{
    if constexpr (OP == Operand::F32) {
        return u32x4{__float_as_uint(v[4 * s + 0]), __float_as_uint(v[4 * s + 1]),
                     __float_as_uint(v[4 * s + 2]), __float_as_uint(v[4 * s + 3])};
    } else {
        return u32x4{pack2<OP>(v[8 * s + 0], v[8 * s + 1]), pack2<OP>(v[8 * s + 2], v[8 * s + 3]),
                     pack2<OP>(v[8 * s + 4], v[8 * s + 5]), pack2<OP>(v[8 * s + 6], v[8 * s + 7])};
    }
}

// acc += A_op * B_op for one slot. Lane l of A_op gives row l%32 of the
// product, lane l of B_op gives column l%32; both carry the same k values.
// For fp32 the slot's four k-pairs go to the four chains acc[0..3].
template <Operand OP> HM_DEV void mma(const u32x4& a, const u32x4& b, f32x16 (&acc)[OperandTraits<OP>::kChains])
{
    if constexpr (OP == Operand::F16) {
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                        __builtin_bit_cast(f16x8, b), acc[0], 0, 0, 0);
    } else if constexpr (OP == Operand::BF16) {
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                         __builtin_bit_cast(bf16x8, b), acc[0], 0, 0, 0);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            acc[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[i]), __uint_as_float(b[i]), acc[i], 0, 0, 0);
    }
}

// One 16-bit MFMA: acc + A_op * B_op.
template <Operand OP> HM_DEV f32x16 mma1(const u32x4& a, const u32x4& b, const f32x16& acc)
{
    if constexpr (OP == Operand::F16)
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), acc, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}

// Sum of the chains, in a fixed pairwise order.
template <int NC> HM_DEV f32x16 chain_sum(const f32x16 (&acc)[NC])
{
    if constexpr (NC == 1) return acc[0];
    else return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

// DPP quad permutations: partner lane t^1 and t^2 within each group of four.
HM_DEV uint32_t dpp_xor1(uint32_t v) { return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false); }
HM_DEV uint32_t dpp_xor2(uint32_t v) { return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false); }
HM_DEV float dpp_xor1f(float v) { return __uint_as_float(dpp_xor1(__float_as_uint(v))); }
HM_DEV float dpp_xor2f(float v) { return __uint_as_float(dpp_xor2(__float_as_uint(v))); }

// 4x4 transpose across a lane quad, 16-bit values. Lane t enters with row t
// (cols 0..3 as two packed words) and leaves with column t (rows 0..3).
HM_DEV u32x2 quad_transpose16(uint32_t d0, uint32_t d1, int t)
{
    const bool odd = t & 1;
    const uint32_t p0 = dpp_xor1(d0), p1 = dpp_xor1(d1);
    // even lane keeps (own.lo, partner.lo), odd lane (partner.hi, own.hi)
    const uint32_t n0 = odd ? __builtin_amdgcn_perm(d0, p0, 0x07060302u) : __builtin_amdgcn_perm(p0, d0, 0x05040100u);
    const uint32_t n1 = odd ? __builtin_amdgcn_perm(d1, p1, 0x07060302u) : __builtin_amdgcn_perm(p1, d1, 0x05040100u);
    const bool hi = t & 2;
    const uint32_t r = dpp_xor2(hi ? n0 : n1);
    return u32x2{hi ? r : n0, hi ? n1 : r};
}

// The same transpose for fp32 values.
HM_DEV f32x4 quad_transpose32(const f32x4& c, int t)
{
    const bool odd = t & 1;
    const float r0 = dpp_xor1f(odd ? c[0] : c[1]);
    const float r1 = dpp_xor1f(odd ? c[2] : c[3]);
    const f32x4 n = odd ? f32x4{r0, c[1], r1, c[3]} : f32x4{c[0], r0, c[2], r1};
    const bool hi = t & 2;
    const float q0 = dpp_xor2f(hi ? n[0] : n[2]);
    const float q1 = dpp_xor2f(hi ? n[1] : n[3]);
    return hi ? f32x4{q0, q1, n[2], n[3]} : f32x4{n[0], n[1], q0, q1};
}

HM_DEV float wave_max(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}

HM_DEV float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// Normalisation of an fp32-operand tile without rounding it. The step is
// homogeneous: with X = Y / rho, one step X <- aX + (bA + cA^2)X is
// Y <- aY + ((b / rho^2) A_Y + (c / rho^4) A_Y^2) Y with A_Y = Y Y^T, and
// Y_K / rho = X_K. So the tile is scaled by a power of two only (exact), to
// Y with ||Y||_F^2 = m in [1, 4), and rho^2 = m goes into the coefficients
// and the output factor; the normalised tile itself is never rounded. The
// coefficients b / m and c / m^2 are carried as unevaluated sums hi + lo of
// two fp32 numbers (formed in fp64), so that they are exact to about 2^-48
// and the polynomial is the one the caller asked for.
// `ss` is the tile's sum of squares (a normal fp32 number, or 0: then
// Phi_K = 0 and everything here is 0).
struct ExactNorm {
    float scale;   // 2^-e, with ss = m 4^e
    float bh, bl;  // b / m = bh + bl
    float ch, cl;  // c / m^2 = ch + cl
    float out;     // 1 / sqrt(m)
};
HM_DEV ExactNorm exact_norm(float ss, float b, float c)
{
    if (!(ss > 0.f)) return ExactNorm{0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const uint32_t sb = __float_as_uint(ss);
    const int e = ((int)(sb >> 23) - 127) >> 1;
    const double m = (double)__uint_as_float(sb - ((uint32_t)(2 * e) << 23));
    const double bd = (double)b / m, cd = (double)c / (m * m);
    const float bh = (float)bd, ch = (float)cd;
    return ExactNorm{ldexpf(1.f, -e), bh, (float)(bd - (double)bh), ch, (float)(cd - (double)ch),
                     (float)(1.0 / sqrt(m))};
}

// b' G + c' Q with b' = bh + bl and c' = ch + cl (the correction terms first)
HM_DEV float poly2(const ExactNorm& n, float g, float q)
{
    return fmaf(n.ch, q, fmaf(n.bh, g, fmaf(n.bl, g, n.cl * q)));
}

// Four consecutive elements of row `gr`, columns gc..gc+3, widened to fp32;
// zero outside the matrix (the zero padding of the tiling operator).
template <Storage ST>
HM_DEV f32x4 load4(const void* base, int64_t gr, int64_t gc, int64_t ld, int64_t rows, int64_t cols, bool vec)
{
    if constexpr (ST == Storage::BF16) {
        const uint16_t* p = static_cast<const uint16_t*>(base) + gr * ld + gc;
        if (vec) {
            const u32x2 w = *reinterpret_cast<const u32x2*>(p);
            return f32x4{__uint_as_float(w[0] << 16), __uint_as_float(w[0] & 0xffff0000u),
                         __uint_as_float(w[1] << 16), __uint_as_float(w[1] & 0xffff0000u)};
        }
        f32x4 r = {0.f, 0.f, 0.f, 0.f};
        if (gr < rows) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (gc + e < cols) r[e] = __uint_as_float(((uint32_t)p[e]) << 16);
        }
        return r;
    } else {
        const float* p = static_cast<const float*>(base) + gr * ld + gc;
        if (vec) return *reinterpret_cast<const f32x4*>(p);
        f32x4 r = {0.f, 0.f, 0.f, 0.f};
        if (gr < rows) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (gc + e < cols) r[e] = p[e];
        }
        return r;
    }
}

// The values a store4 of v leaves in memory (bf16: rounded to nearest even).
template <Storage ST>
HM_DEV f32x4 stored4(const f32x4& v)
{
    if constexpr (ST == Storage::BF16) {
        f32x4 r;
#pragma unroll
        for (int e = 0; e < 4; ++e) r[e] = (float)(__bf16)v[e];
        return r;
    } else {
        return v;
    }
}

// Store four values (rounded to nearest even for bf16), dropping the
// padding (inverse tiling operator).
template <Storage ST>
HM_DEV void store4(void* base, int64_t gr, int64_t gc, int64_t ld, int64_t rows, int64_t cols, bool vec, const f32x4& v)
{
    if constexpr (ST == Storage::BF16) {
        uint16_t* p = static_cast<uint16_t*>(base) + gr * ld + gc;
        const uint32_t w0 = pack2<Operand::BF16>(v[0], v[1]);
        const uint32_t w1 = pack2<Operand::BF16>(v[2], v[3]);
        if (vec) {
            *reinterpret_cast<u32x2*>(p) = u32x2{w0, w1};
            return;
        }
        if (gr < rows) {
            const uint16_t h[4] = {(uint16_t)(w0 & 0xffffu), (uint16_t)(w0 >> 16), (uint16_t)(w1 & 0xffffu),
                                   (uint16_t)(w1 >> 16)};
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (gc + e < cols) p[e] = h[e];
        }
    } else {
        float* p = static_cast<float*>(base) + gr * ld + gc;
        if (vec) {
            *reinterpret_cast<f32x4*>(p) = v;
            return;
        }
        if (gr < rows) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (gc + e < cols) p[e] = v[e];
        }
    }
}

}  // namespace dev
}  // namespace himuon
