// Fused tiled Newton–Schulz kernels for gfx950 (MI355X).
//
// One launch evaluates Phi_K (Sec. 2.2, eqs. ns_iteration / ns_quintic /
// phi_k_def) on every tile of a chunk of the batched tile set (Sec. 4.1,
// eq. tiled_ns; Sec. 4.4.2, cross-layer batching). Each tile is read from HBM
// once, kept on chip (registers + LDS) for all K steps, and written once.
//
// Data layout on chip. A tile is a grid of 32x32 blocks (NB = T/32 per side).
// A wave owns RB consecutive block rows ("row blocks") of its tile and keeps
// them as fp32 v_mfma 32x32 accumulators. In that accumulator layout lane l
// holds, for block column q, the 16 values
//     row  = l % 32,
//     cols = 8g + 4(l/32) + e        (g, e = 0..3; register 4g+e),
// i.e. a piece of one row ("row piece"). Because A = X X^T and A^2 = A A^T
// contract over columns, a row piece is already a valid MFMA operand for
// both Gram-type products, and with the operands in the order
// (other rows, own rows) the MFMA result is again a row piece of the output
// (A is symmetric). No transpose is needed for those two products.
//
// The third product, B X, contracts X over rows. Its MFMA operand is a
// "column piece" of X (one column, rows in the same 8g+4h+e pattern); every
// step writes X once more to LDS in that layout, after a 4x4 transpose
// inside each lane quad done with DPP (no LDS traffic for the transpose).
//
// Epilogues. With 16-bit operands they live in the accumulators: the A^2
// accumulator starts from (b/c)·A and is scaled by c, giving B = bA + cA^2
// from fp32 A; the product accumulator starts from a·X (fp32 master copy),
// giving aX + BX. With fp32 operands every accumulator starts at zero (four
// chains each) and B = fma(c, A^2, bA), X = fma(a, X, BX) are formed once at
// the end, which keeps large partial sums out of the fp32 rounding walk.
// Operands are rounded once (fp16 or bf16, round to nearest even) or stay fp32.
//
// LDS holds, per tile, one operand matrix of row pieces ("xr", only when a
// tile is split over several waves; it carries X and then A) and one of
// column pieces ("xc"), both as 16-byte-per-lane slots in lane order so
// every LDS read and most writes are conflict-free 128-bit accesses.
#include "himuon_internal.h"

#include <atomic>
#include <type_traits>
#include <math.h>

namespace himuon {
namespace {

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

constexpr int kThreads = 256;  // four waves per workgroup

// T: tile size; RB: 32-row blocks per wave. A tile is spread over
// WT = T/(32 RB) waves, and a workgroup of four waves runs 4/WT tiles.
template <int T, int RB, Storage ST, Operand OP>
__global__ void __launch_bounds__(kThreads) ns_tiled_kernel(const KernelArgs args)
{
    constexpr int NB = T / 32;
    constexpr int WT = NB / RB;
    static_assert(NB % RB == 0 && WT >= 1 && WT <= 4, "tile split");
    constexpr int TPW = 4 / WT;
    constexpr int S = OperandTraits<OP>::kSlots;
    constexpr int NC = OperandTraits<OP>::kChains;
    constexpr int MAT = NB * NB * S * 64;  // 16-byte slots in one operand matrix
    constexpr bool SHARED_ROWS = WT > 1;

    __shared__ u32x4 s_xr[SHARED_ROWS ? TPW * MAT : 1];
    __shared__ u32x4 s_xc[TPW * MAT];
    __shared__ float s_red[2][4];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int tslot = wave / WT;
    const int p0 = (wave % WT) * RB;  // first owned row block
    const int li = lane & 31, lh = lane >> 5;
    u32x4* const xr = s_xr + (SHARED_ROWS ? tslot * MAT : 0);
    u32x4* const xc = s_xc + tslot * MAT;

    const int64_t n_tiles = args.tile_end - args.tile_begin;
    const int64_t n_groups = (n_tiles + TPW - 1) / TPW;

    for (int64_t grp = blockIdx.x; grp < n_groups; grp += gridDim.x) {
        const int64_t local = grp * TPW + tslot;
        const bool valid = local < n_tiles;
        if constexpr (!SHARED_ROWS || TPW == 1) {
            if (!valid) continue;  // no workgroup barrier depends on this wave
        }
        const int64_t tile = args.tile_begin + (valid ? local : 0);

        // matrix owning the tile: last descriptor with tile_begin <= tile
        int lo = 0, hi = args.n_mats - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (args.descs[mid].tile_begin <= tile) lo = mid;
            else hi = mid - 1;
        }
        lo = __builtin_amdgcn_readfirstlane(lo);
        const MatDesc& d = args.descs[lo];
        const int64_t lt = tile - d.tile_begin;
        const int64_t tr = lt / d.tiles_c;
        const int64_t row0 = tr * T, col0 = (lt - tr * d.tiles_c) * T;
        const bool full = row0 + T <= d.rows && col0 + T <= d.cols;
        const bool vin = full && (d.flags & MAT_VEC_IN);
        const bool vout = full && (d.flags & MAT_VEC_OUT);
        const int64_t rows_eff = valid ? d.rows : 0;  // an idle wave reads zeros

        // ---- gather the tile (zero padded) into fp32 row pieces
        f32x16 X[RB][NB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int64_t gr = row0 + 32 * (p0 + rb) + li;
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const f32x4 v = load4<ST>(d.in, gr, col0 + 32 * q + 8 * g + 4 * lh, d.ld_in, rows_eff, d.cols, vin);
                    X[rb][q][4 * g + 0] = v[0];
                    X[rb][q][4 * g + 1] = v[1];
                    X[rb][q][4 * g + 2] = v[2];
                    X[rb][q][4 * g + 3] = v[3];
                }
        }

        // ---- X_0 = S / ||S||_F, after an exact power-of-two pre-scale so the
        //      fp32 sum of squares neither overflows nor underflows
        float mx = 0.f;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int v = 0; v < 16; ++v) mx = fmaxf(mx, fabsf(X[rb][q][v]));
        mx = wave_max(mx);
        if constexpr (SHARED_ROWS) {
            if (lane == 0) s_red[0][wave] = mx;
            __syncthreads();
            mx = s_red[0][tslot * WT];
#pragma unroll
            for (int w = 1; w < WT; ++w) mx = fmaxf(mx, s_red[0][tslot * WT + w]);
        }
        int ex = 0;
        (void)frexpf(mx, &ex);
        const float s1 = ldexpf(1.f, -(ex / 2)), s2 = ldexpf(1.f, -(ex - ex / 2));
        float ss = 0.f;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const float y = X[rb][q][v] * s1 * s2;
                    X[rb][q][v] = y;
                    ss = fmaf(y, y, ss);
                }
        ss = wave_sum(ss);
        if constexpr (SHARED_ROWS) {
            if (lane == 0) s_red[1][wave] = ss;
            __syncthreads();
            ss = s_red[1][tslot * WT];
#pragma unroll
            for (int w = 1; w < WT; ++w) ss += s_red[1][tslot * WT + w];
        }
        const float inv = ss > 0.f ? 1.f / sqrtf(ss) : 0.f;  // Phi_K(0) = 0
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int q = 0; q < NB; ++q) X[rb][q] *= inv;

        // ---- K Newton–Schulz steps, all on chip
        const int t4 = li & 3, quad = li >> 2;
        const int xg = quad >> 1, xh = quad & 1;  // row group of this quad in a block
        for (int k = 0; k < args.K; ++k) {
            u32x4 Xop[RB][NB][S];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int q = 0; q < NB; ++q)
#pragma unroll
                    for (int s = 0; s < S; ++s) Xop[rb][q][s] = make_slot<OP>(X[rb][q], s);

            if constexpr (SHARED_ROWS) {
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int q = 0; q < NB; ++q)
#pragma unroll
                        for (int s = 0; s < S; ++s) xr[(((p0 + rb) * NB + q) * S + s) * 64 + lane] = Xop[rb][q][s];
            }
            // column pieces of X for the B X product
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                const int Q = p0 + rb;
#pragma unroll
                for (int N = 0; N < NB; ++N)
#pragma unroll
                    for (int gp = 0; gp < 4; ++gp) {
                        const int lane_dst = xh * 32 + 8 * gp + 4 * lh + t4;
                        if constexpr (OP == Operand::F32) {
                            const f32x4 c = {X[rb][N][4 * gp + 0], X[rb][N][4 * gp + 1], X[rb][N][4 * gp + 2],
                                             X[rb][N][4 * gp + 3]};
                            const f32x4 o = quad_transpose32(c, t4);
                            xc[((Q * NB + N) * S + xg) * 64 + lane_dst] = __builtin_bit_cast(u32x4, o);
                        } else {
                            const u32x4& w = Xop[rb][N][gp >> 1];
                            const u32x2 o = quad_transpose16(w[(gp & 1) * 2], w[(gp & 1) * 2 + 1], t4);
                            u32x2* dst = reinterpret_cast<u32x2*>(&xc[((Q * NB + N) * S + (xg >> 1)) * 64 + lane_dst]);
                            dst[xg & 1] = o;
                        }
                    }
            }
            if constexpr (SHARED_ROWS) __syncthreads();

            // A = X X^T as row pieces of the owned rows
            f32x16 G[RB][NB];
            {
                f32x16 Gc[RB][NB][NC];
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int J = 0; J < NB; ++J)
#pragma unroll
                        for (int ch = 0; ch < NC; ++ch) Gc[rb][J][ch] = f32x16{};
#pragma unroll
                for (int J = 0; J < NB; ++J)
#pragma unroll
                    for (int q = 0; q < NB; ++q)
#pragma unroll
                        for (int s = 0; s < S; ++s) {
                            u32x4 opa;
                            if constexpr (SHARED_ROWS) opa = xr[((J * NB + q) * S + s) * 64 + lane];
                            else opa = Xop[J][q][s];
#pragma unroll
                            for (int rb = 0; rb < RB; ++rb) mma<OP>(opa, Xop[rb][q][s], Gc[rb][J]);
                        }
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int J = 0; J < NB; ++J) G[rb][J] = chain_sum<NC>(Gc[rb][J]);
            }

            // B = bA + cA^2. 16-bit operands: accumulated in place as
            // c((b/c)A + A A^T). fp32 operands: A^2 in zero-started chains,
            // then one fused b*A + c*A^2 from the fp32 A (no large partial sums).
            if (args.c != 0.f) {
                u32x4 Aop[RB][NB][S];
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int J = 0; J < NB; ++J) {
#pragma unroll
                        for (int s = 0; s < S; ++s) Aop[rb][J][s] = make_slot<OP>(G[rb][J], s);
                        if constexpr (OP != Operand::F32) G[rb][J] *= args.b_over_c;
                    }
                if constexpr (SHARED_ROWS) {
                    __syncthreads();  // every wave is done reading X from xr
#pragma unroll
                    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                        for (int J = 0; J < NB; ++J)
#pragma unroll
                            for (int s = 0; s < S; ++s) xr[(((p0 + rb) * NB + J) * S + s) * 64 + lane] = Aop[rb][J][s];
                    __syncthreads();
                }
                f32x16 Gc[RB][NB][NC];
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int J = 0; J < NB; ++J) {
                        if constexpr (OP == Operand::F32) Gc[rb][J][0] = f32x16{};
                        else Gc[rb][J][0] = G[rb][J];
#pragma unroll
                        for (int ch = 1; ch < NC; ++ch) Gc[rb][J][ch] = f32x16{};
                    }
#pragma unroll
                for (int J = 0; J < NB; ++J)
#pragma unroll
                    for (int q = 0; q < NB; ++q)
#pragma unroll
                        for (int s = 0; s < S; ++s) {
                            u32x4 opa;
                            if constexpr (SHARED_ROWS) opa = xr[((J * NB + q) * S + s) * 64 + lane];
                            else opa = Aop[J][q][s];
#pragma unroll
                            for (int rb = 0; rb < RB; ++rb) mma<OP>(opa, Aop[rb][q][s], Gc[rb][J]);
                        }
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int J = 0; J < NB; ++J) {
                        const f32x16 sq = chain_sum<NC>(Gc[rb][J]);
                        if constexpr (OP == Operand::F32) {
#pragma unroll
                            for (int v = 0; v < 16; ++v) G[rb][J][v] = fmaf(args.c, sq[v], args.b * G[rb][J][v]);
                        } else {
                            G[rb][J] = sq * args.c;
                        }
                    }
            } else {
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int J = 0; J < NB; ++J) G[rb][J] *= args.b;
            }

            // X <- aX + B X
            u32x4 Bop[RB][NB][S];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int Q = 0; Q < NB; ++Q)
#pragma unroll
                    for (int s = 0; s < S; ++s) Bop[rb][Q][s] = make_slot<OP>(G[rb][Q], s);
            {
                f32x16 Pc[RB][NB][NC];
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int N = 0; N < NB; ++N) {
                        if constexpr (OP == Operand::F32) Pc[rb][N][0] = f32x16{};
                        else Pc[rb][N][0] = X[rb][N] * args.a;
#pragma unroll
                        for (int ch = 1; ch < NC; ++ch) Pc[rb][N][ch] = f32x16{};
                    }
#pragma unroll
                for (int N = 0; N < NB; ++N)
#pragma unroll
                    for (int Q = 0; Q < NB; ++Q)
#pragma unroll
                        for (int s = 0; s < S; ++s) {
                            const u32x4 opa = xc[((Q * NB + N) * S + s) * 64 + lane];
#pragma unroll
                            for (int rb = 0; rb < RB; ++rb) mma<OP>(opa, Bop[rb][Q][s], Pc[rb][N]);
                        }
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int N = 0; N < NB; ++N) {
                        const f32x16 bx = chain_sum<NC>(Pc[rb][N]);
                        if constexpr (OP == Operand::F32) {
#pragma unroll
                            for (int v = 0; v < 16; ++v) X[rb][N][v] = fmaf(args.a, X[rb][N][v], bx[v]);
                        } else {
                            X[rb][N] = bx;
                        }
                    }
            }
            if constexpr (SHARED_ROWS) __syncthreads();  // xr / xc are rewritten next step
        }

        // ---- write back the unpadded part
        if (valid) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                const int64_t gr = row0 + 32 * (p0 + rb) + li;
#pragma unroll
                for (int q = 0; q < NB; ++q)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const f32x4 v = {X[rb][q][4 * g + 0], X[rb][q][4 * g + 1], X[rb][q][4 * g + 2],
                                         X[rb][q][4 * g + 3]};
                        store4<ST>(d.out, gr, col0 + 32 * q + 8 * g + 4 * lh, d.ld_out, d.rows, d.cols, vout, v);
                    }
            }
        }
    }
}

// ------------------------------------------------ fp16-operand kernel
//
// Same tile map, restructured so that almost no vector-ALU work is left in
// the K loop. The state is Z = X |c|^(1/4) (exact rescaling of the iterate),
// for which one step of eq. (ns_iteration) reads
//     Z <- a Z + P Z,   P = sigma H (H + sigma b' I),   H = Z Z^T,
// with b' = b / sqrt|c| and sigma = sign(c): the c-coefficient becomes +-1
// and b' moves onto the diagonal of an MFMA operand, so the only per-element
// multiply left is the fp32 a*Z that seeds the product accumulator (the a*Z
// term stays in fp32, which keeps rounding out of the directions the
// iteration amplifies). The normalisation multiplies by |c|^(1/4) and the
// store by |c|^(-1/4). c = 0 takes P = b H.
//
// Z is shared through one row-major fp16 copy of the tile (see kRowStride).
// Gram operands of the other waves' rows are read from it as row pieces; the
// B X operand (column pieces of Z) comes from it through ds_read_b64_tr_b16,
// which returns in every lane quad a 4x4 transpose of four rows supplied by
// the other lanes of its 16-lane group. H is shared through 16-byte
// lane-ordered slots. A wave works on the blocks of its row in the rotated
// order J = (p + j) mod NB, so its own row blocks come from registers.
//
// Tiles are processed in rounds; the HBM loads of a wave's next tile are
// issued before the current tile is written back.

// 64-bit DPP move (both halves with the same control).
template <int CTRL> HM_DEV double dpp_f64(double v)
{
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)u, CTRL, 0xF, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, false);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

HM_DEV double readlane_f64(double v, int l)
{
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Sum over the 64 lanes in a fixed order: butterflies inside each 16-lane
// row (quad swaps, half-row and row mirrors), then the four row sums.
HM_DEV double wave_sum_f64(double v)
{
    v += dpp_f64<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp_f64<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp_f64<0x141>(v);  // row_half_mirror
    v += dpp_f64<0x140>(v);  // row_mirror
    return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

// Matrix owning `tile`, searching from `hint` (the tiles one wave visits only
// grow, so the owner of an earlier tile is a lower bound).
HM_DEV int find_matrix_from(const KernelArgs& args, int64_t tile, int hint)
{
    if (hint + 1 >= args.n_mats || args.descs[hint + 1].tile_begin > tile) return hint;
    int lo = hint + 1, hi = args.n_mats - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (args.descs[mid].tile_begin <= tile) lo = mid;
        else hi = mid - 1;
    }
    return __builtin_amdgcn_readfirstlane(lo);
}

// Four consecutive bf16 elements of row gr (columns gc..gc+3) as two packed
// words, zero outside the matrix (the zero padding of the tiling operator).
HM_DEV u32x2 load_bf16x4(const void* base, int64_t gr, int64_t gc, int64_t ld, int64_t rows, int64_t cols, bool vec)
{
    const uint16_t* p = static_cast<const uint16_t*>(base) + gr * ld + gc;
    if (vec) return *reinterpret_cast<const u32x2*>(p);
    uint32_t h[4] = {0u, 0u, 0u, 0u};
    if (gr < rows) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (gc + e < cols) h[e] = p[e];
    }
    return u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
}

HM_DEV u32x2 tr_read(const uint8_t* ptr)
{
    typedef short s4 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) s4* lds_s4p;
    const s4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4p)(ptr));
    return __builtin_bit_cast(u32x2, v);
}

// Row-major fp16 copy of Z. Bytes per row: an odd multiple of 64, so the
// eight consecutive rows a transposing read touches (64 bytes each) fall on
// four distinct quarters of the 256-byte bank space, twice each. Within each
// 64-byte segment (32 columns) the 8-byte chunk c of row r sits at chunk
// c ^ 2((r >> 2) & 3): rows r, r+4, ..., r+28 share a quarter, and the XOR
// spreads their row-piece chunks (2g + lh) over all eight chunks, so
// row-piece reads and writes (32 rows x 16 bytes) are conflict-free as well.
template <int T> constexpr int kRowStride = ((2 * T / 64) % 2 == 1) ? 2 * T : 2 * T + 64;

// A wave that owns two row blocks of a 128-tile needs more than 256
// registers; everything else runs two waves per SIMD.
template <int T, int RB> constexpr int kF16MinBlocks = (T / 32) / RB == 2 ? 1 : 2;

// CMODE: 0 for c > 0, 1 for c < 0, 2 for c = 0 (sign(c) and the c = 0
// shortcut are compile-time, so no branch of the K loop is if-converted).
// RB: 32-row blocks owned by one wave; a tile is spread over NB / RB waves.
// Every operand read from LDS feeds RB MFMAs.
template <int T, int RB, int CMODE>
__global__ void __launch_bounds__(kThreads, (kF16MinBlocks<T, RB>)) ns_tiled_f16_kernel(const KernelArgs args)
{
    constexpr Storage ST = Storage::BF16;
    constexpr Operand OP = Operand::F16;
    constexpr int NB = T / 32;      // row blocks per tile
    constexpr int WT = NB / RB;     // waves per tile
    static_assert(NB % RB == 0 && WT >= 1 && WT <= 4, "tile split");
    constexpr int TPW = 4 / WT;     // tiles per workgroup
    constexpr int S = 2;
    constexpr int MAT = NB * NB * S * 64;  // 16-byte slots of H
    constexpr bool SHARED = WT > 1;
    static_assert(!SHARED || TPW == 1, "a workgroup that shares a tile runs one tile");
    constexpr int NO = NB - RB;     // row blocks owned by the other waves of the tile
    constexpr int NOA = NO > 0 ? NO : 1;
    constexpr int RS = kRowStride<T>;
    constexpr int RM = T * RS;
    constexpr int IT = NB * S;      // k iterations of one product

    __shared__ u32x4 s_slots[SHARED ? TPW * MAT : 1];
    __shared__ __attribute__((aligned(16))) uint8_t s_rm[TPW * RM];
    __shared__ double s_red64[4];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int tslot = wave / WT, p0 = (wave % WT) * RB;
    const int li = lane & 31, lh = lane >> 5;
    u32x4* const slots = s_slots + (SHARED ? tslot * MAT : 0);
    uint8_t* const rm = s_rm + tslot * RM;
    // Row pieces: this lane's columns 32q + 8g + 4lh of row li of a block are
    // chunk 2g + lh of the block's segment, stored at chunk 2(g ^ fl) + lh.
    const int fl = (li >> 2) & 3;
    int rp_off[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) rp_off[g] = li * RS + 16 * (g ^ fl) + 8 * lh;
    // Transposing reads: supplier lane 4q' + m of 16-lane group G addresses
    // row 4(G/2) + m (+ 8x) and logical chunk 4(G%2) + q' of a block segment.
    const int grp16 = lane >> 4;
    int tr_off[2];
#pragma unroll
    for (int x = 0; x < 2; ++x) {
        const int row = 8 * x + 4 * (grp16 >> 1) + ((lane & 15) >> 2);
        const int chunk = 4 * (grp16 & 1) + (lane & 3);
        tr_off[x] = row * RS + 8 * (chunk ^ (2 * ((row >> 2) & 3)));
    }
    // A diagonal block holds row li's column 8g + 4lh + e in register 4g + e,
    // so the diagonal entry of this lane (if any) is register vdiag.
    const int vdiag = (lh == ((li >> 2) & 1)) ? 4 * (li >> 3) + (li & 3) : -1;
    // the row blocks owned by the other waves, in rotated order: H slots and
    // the rows of the row-major copy
    u32x4* sl_row[NOA];
    const uint8_t* rm_row[NOA];
#pragma unroll
    for (int jo = 0; jo < NOA; ++jo) {
        sl_row[jo] = slots + (((p0 + RB + jo) % NB) * NB * S) * 64 + lane;
        rm_row[jo] = rm + 32 * ((p0 + RB + jo) % NB) * RS;
    }
    auto rowpiece = [&](const uint8_t* blockrow, int q, int s) -> u32x4 {
        const u32x2 lo = *reinterpret_cast<const u32x2*>(blockrow + rp_off[2 * s] + 64 * q);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(blockrow + rp_off[2 * s + 1] + 64 * q);
        return u32x4{lo[0], lo[1], hi[0], hi[1]};
    };

    const int64_t n_tiles = args.tile_end - args.tile_begin;

    // Tile placement. The tile of the next round is located, and its HBM
    // loads are issued, before the current tile is written back.
    struct TileLoc {
        const MatDesc* d;
        int64_t row0, col0;
        bool vin, vout;
    };
    int mhint = 0;
    auto locate = [&](int64_t local, TileLoc& L) {
        const int64_t tile = args.tile_begin + local;
        mhint = find_matrix_from(args, tile, mhint);
        L.d = &args.descs[mhint];
        const int64_t lt = tile - L.d->tile_begin;
        const int64_t tr = lt / L.d->tiles_c;
        L.row0 = tr * T;
        L.col0 = (lt - tr * L.d->tiles_c) * T;
        const bool full = L.row0 + T <= L.d->rows && L.col0 + T <= L.d->cols;
        L.vin = full && (L.d->flags & MAT_VEC_IN);
        L.vout = full && (L.d->flags & MAT_VEC_OUT);
    };
    // HBM traffic in whole row segments: a lane moves 16 bytes (8 bf16), a
    // row takes LPR lanes and one wave instruction RPI rows. The wave's own
    // RB row blocks take NI instructions; the row pieces are then reshaped
    // through the wave's own rows of the row-major copy.
    constexpr int LPR = T / 8;
    constexpr int RPI = 64 / LPR;
    constexpr int NI = 32 * RB / RPI;
    const int io_row = lane / LPR, io_cc = lane % LPR;  // row within an instruction, 16-byte chunk
    u32x4 raw[NI];
    auto issue_loads = [&](const TileLoc& L) {
        const int64_t gr0 = L.row0 + 32 * p0 + io_row;
        const int64_t gc = L.col0 + 8 * io_cc;
        if (L.vin) {  // whole tile inside, 16-byte aligned: straight vector loads
            const gbl_u32x4* src = (const gbl_u32x4*)(static_cast<const uint16_t*>(L.d->in) + gr0 * L.d->ld_in + gc);
            const int64_t step = (int64_t)RPI * L.d->ld_in / 8;  // u32x4 per RPI rows
#pragma unroll
            for (int i = 0; i < NI; ++i) raw[i] = src[i * step];
        } else {
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                const int64_t gr = gr0 + RPI * i;
                const uint16_t* ptr = static_cast<const uint16_t*>(L.d->in) + gr * L.d->ld_in + gc;
                uint32_t h[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
                if (gr < L.d->rows) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (gc + e < L.d->cols) h[e] = ptr[e];
                }
                raw[i] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
            }
        }
    };
    // byte offset of the 16-byte chunk io_cc of tile row `row` in the row-major copy
    auto io_lds = [&](int row) -> int {
        return row * RS + 64 * (io_cc >> 2) + 8 * ((2 * (io_cc & 3)) ^ (2 * ((row >> 2) & 3)));
    };

    int64_t local = (int64_t)blockIdx.x * TPW + tslot;
    if (local >= n_tiles) return;  // uniform over the waves that share a tile
    TileLoc cur;
    locate(local, cur);
    issue_loads(cur);

    for (;;) {
        const int64_t nlocal = local + (int64_t)gridDim.x * TPW;
        const bool has_next = nlocal < n_tiles;
        TileLoc nxt = cur;
        if (has_next) locate(nlocal, nxt);

        // own rows into the row-major copy, then back as row pieces (bf16 -> fp32);
        // only this wave touches these rows until its first step's barrier
#pragma unroll
        for (int i = 0; i < NI; ++i) *reinterpret_cast<u32x4*>(rm + io_lds(32 * p0 + RPI * i + io_row)) = raw[i];
        f32x16 Z[RB][NB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const u32x2 w = *reinterpret_cast<const u32x2*>(rm + 32 * (p0 + rb) * RS + rp_off[g] + 64 * q);
                    Z[rb][q][4 * g + 0] = __uint_as_float(w[0] << 16);
                    Z[rb][q][4 * g + 1] = __uint_as_float(w[0] & 0xffff0000u);
                    Z[rb][q][4 * g + 2] = __uint_as_float(w[1] << 16);
                    Z[rb][q][4 * g + 3] = __uint_as_float(w[1] & 0xffff0000u);
                }

        // Z_0 = |c|^(1/4) S / ||S||_F. The sum of squares is taken in fp64,
        // whose range covers every bf16 tile; the scale is applied as an fp32
        // mantissa times an exact power of two.
        double ss = 0.0;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int v = 0; v < 16; ++v) ss = fma((double)Z[rb][q][v], (double)Z[rb][q][v], ss);
        ss = wave_sum_f64(ss);
        if constexpr (SHARED) {
            if (lane == 0) s_red64[wave] = ss;
            __syncthreads();
            ss = s_red64[tslot * WT];
#pragma unroll
            for (int w = 1; w < WT; ++w) ss += s_red64[tslot * WT + w];
        }
        {
            const double nrm = sqrt(ss);
            int ex = 0;
            const float mant = nrm == 0.0 ? 0.f : (float)frexp((double)args.zscale / nrm, &ex);  // Phi_K(0) = 0
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int q = 0; q < NB; ++q)
#pragma unroll
                    for (int v = 0; v < 16; ++v) Z[rb][q][v] = ldexpf(Z[rb][q][v] * mant, ex);
        }

        // One Newton-Schulz step.
        auto ns_step = [&]() {
            u32x4 Zop[RB][NB][S];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int q = 0; q < NB; ++q)
#pragma unroll
                    for (int s = 0; s < S; ++s) Zop[rb][q][s] = make_slot<OP>(Z[rb][q], s);
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int N = 0; N < NB; ++N)
#pragma unroll
                    for (int g = 0; g < 4; ++g)
                        *reinterpret_cast<u32x2*>(rm + 32 * (p0 + rb) * RS + rp_off[g] + 64 * N) =
                            u32x2{Zop[rb][N][g >> 1][(g & 1) * 2], Zop[rb][N][g >> 1][(g & 1) * 2 + 1]};
            if constexpr (SHARED) __syncthreads();

            // H = Z Z^T; G[rb][j] is the row piece of block (p0 + rb, (p0 + j) mod NB).
            // Iteration it = (q, s) reads the other waves' row pieces (q, s) from
            // the row-major copy; those of iteration it + 1 are requested before
            // its MFMAs issue.
            f32x16 G[RB][NB];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int j = 0; j < NB; ++j) G[rb][j] = f32x16{};
            {
                u32x4 nxt_op[NOA];
                if constexpr (NO > 0) {
#pragma unroll
                    for (int jo = 0; jo < NO; ++jo) nxt_op[jo] = rowpiece(rm_row[jo], 0, 0);
                }
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    const int q = it / S, s = it % S;
                    u32x4 cur_op[NOA];
#pragma unroll
                    for (int jo = 0; jo < NOA; ++jo) cur_op[jo] = nxt_op[jo];
                    if constexpr (NO > 0) {
                        if (it + 1 < IT) {
#pragma unroll
                            for (int jo = 0; jo < NO; ++jo) nxt_op[jo] = rowpiece(rm_row[jo], (it + 1) / S, (it + 1) % S);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of these MFMAs
#pragma unroll
                    for (int j = 0; j < NB; ++j) {
                        const u32x4 opa = j < RB ? Zop[j < RB ? j : 0][q][s] : cur_op[j < RB ? 0 : j - RB];
#pragma unroll
                        for (int rb = 0; rb < RB; ++rb) G[rb][j] = mma1<OP>(opa, Zop[rb][q][s], G[rb][j]);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }

            u32x4 Pop[RB][NB][S];  // own rows of P (rotated k-blocks), fp16
            if constexpr (CMODE != 2) {
                u32x4 Hop[RB][NB][S], Q0[RB][S];
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
                    for (int j = 0; j < NB; ++j)
#pragma unroll
                        for (int s = 0; s < S; ++s) Hop[rb][j][s] = make_slot<OP>(G[rb][j], s);
                    f32x16 gd = G[rb][rb];  // H + sigma b' I on the diagonal block (p0 + rb, p0 + rb)
#pragma unroll
                    for (int v = 0; v < 16; ++v) gd[v] += v == vdiag ? args.bq : 0.f;
#pragma unroll
                    for (int s = 0; s < S; ++s) Q0[rb][s] = make_slot<OP>(gd, s);
                }
                if constexpr (SHARED) {
                    // the H slots were last read before the previous step's final barrier
#pragma unroll
                    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                        for (int j = 0; j < NB; ++j)
#pragma unroll
                            for (int s = 0; s < S; ++s)
                                slots[(((p0 + rb) * NB + (p0 + j) % NB) * S + s) * 64 + lane] = Hop[rb][j][s];
                    __syncthreads();
                }
                // P' = H (H + sigma b' I): acc[rb][j] is block (p0 + rb, (p0 + j) mod NB);
                // iteration it = (jk, s) runs over the rotated k-blocks (p0 + jk) mod NB.
                f32x16 acc[RB][NB];
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int j = 0; j < NB; ++j) acc[rb][j] = f32x16{};
                auto h_slot = [&](int jo, int it) -> u32x4 {
                    const int jk = it / S, s = it % S;
                    return sl_row[jo][(((p0 + jk) % NB) * S + s) * 64];
                };
                u32x4 nxt_op[NOA];
                if constexpr (NO > 0) {
#pragma unroll
                    for (int jo = 0; jo < NO; ++jo) nxt_op[jo] = h_slot(jo, 0);
                }
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    const int jk = it / S, s = it % S;
                    u32x4 cur_op[NOA];
#pragma unroll
                    for (int jo = 0; jo < NOA; ++jo) cur_op[jo] = nxt_op[jo];
                    if constexpr (NO > 0) {
                        if (it + 1 < IT) {
#pragma unroll
                            for (int jo = 0; jo < NO; ++jo) nxt_op[jo] = h_slot(jo, it + 1);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int j = 0; j < NB; ++j) {
                        const u32x4 opa = j < RB ? Hop[j < RB ? j : 0][jk][s] : cur_op[j < RB ? 0 : j - RB];
#pragma unroll
                        for (int rb = 0; rb < RB; ++rb) {
                            const u32x4 opb = jk == rb ? Q0[rb][s] : Hop[rb][jk][s];
                            acc[rb][j] = mma1<OP>(opa, opb, acc[rb][j]);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int j = 0; j < NB; ++j)
#pragma unroll
                        for (int s = 0; s < S; ++s) {
                            if constexpr (CMODE == 0) Pop[rb][j][s] = make_slot<OP>(acc[rb][j], s);
                            else Pop[rb][j][s] = make_slot<OP>(-acc[rb][j], s);
                        }
            } else {
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int j = 0; j < NB; ++j)
#pragma unroll
                        for (int s = 0; s < S; ++s) Pop[rb][j][s] = make_slot<OP>(G[rb][j] * args.bq, s);
            }


            // Z <- a Z + P Z; iteration it = (jk, s) needs the column pieces of
            // k-block (p0 + jk) mod NB for every output block N (two transposing
            // reads each), shared by the RB owned row blocks.
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int N = 0; N < NB; ++N) Z[rb][N] *= args.a;
            {
                auto col_piece = [&](int it, int N) -> u32x4 {
                    const int jk = it / S, s = it % S;
                    const uint8_t* const kb = rm + 32 * ((p0 + jk) % NB) * RS + 16 * s * RS + 64 * N;
                    const u32x2 lo = tr_read(kb + tr_off[0]);
                    const u32x2 hi = tr_read(kb + tr_off[1]);
                    return u32x4{lo[0], lo[1], hi[0], hi[1]};
                };
                u32x4 nxt_op[NB];
#pragma unroll
                for (int N = 0; N < NB; ++N) nxt_op[N] = col_piece(0, N);
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    const int jk = it / S, s = it % S;
                    u32x4 cur_op[NB];
#pragma unroll
                    for (int N = 0; N < NB; ++N) cur_op[N] = nxt_op[N];
                    if (it + 1 < IT) {
#pragma unroll
                        for (int N = 0; N < NB; ++N) nxt_op[N] = col_piece(it + 1, N);
                    }
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int N = 0; N < NB; ++N)
#pragma unroll
                        for (int rb = 0; rb < RB; ++rb) Z[rb][N] = mma1<OP>(cur_op[N], Pop[rb][jk][s], Z[rb][N]);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            if constexpr (SHARED) __syncthreads();  // the row-major copy and the H slots are rewritten next step
        };
        for (int k = 0; k < args.K; ++k) ns_step();

        // row pieces (scaled back, rounded to bf16) into the own rows of the
        // row-major copy, then whole row segments to HBM; the next tile's loads
        // are issued in between, once the state registers are free
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const f32x4 v = f32x4{Z[rb][q][4 * g + 0], Z[rb][q][4 * g + 1], Z[rb][q][4 * g + 2],
                                          Z[rb][q][4 * g + 3]} * args.unscale;
                    *reinterpret_cast<u32x2*>(rm + 32 * (p0 + rb) * RS + rp_off[g] + 64 * q) =
                        u32x2{pack2<Operand::BF16>(v[0], v[1]), pack2<Operand::BF16>(v[2], v[3])};
                }
        // (raw is defined on both paths, so the values staged at the top of
        // this round are dead across its steps)
        if (has_next) {
            issue_loads(nxt);
        } else {
#pragma unroll
            for (int i = 0; i < NI; ++i) raw[i] = u32x4{};
        }
        {
            const int64_t gr0 = cur.row0 + 32 * p0 + io_row;
            const int64_t gc = cur.col0 + 8 * io_cc;
            if (cur.vout) {
                gbl_u32x4* dst = (gbl_u32x4*)(static_cast<uint16_t*>(cur.d->out) + gr0 * cur.d->ld_out + gc);
                const int64_t step = (int64_t)RPI * cur.d->ld_out / 8;
#pragma unroll
                for (int i = 0; i < NI; ++i) dst[i * step] = *reinterpret_cast<const u32x4*>(rm + io_lds(32 * p0 + RPI * i + io_row));
            } else {
#pragma unroll
                for (int i = 0; i < NI; ++i) {
                    const u32x4 w = *reinterpret_cast<const u32x4*>(rm + io_lds(32 * p0 + RPI * i + io_row));
                    const int64_t gr = gr0 + RPI * i;
                    uint16_t* ptr = static_cast<uint16_t*>(cur.d->out) + gr * cur.d->ld_out + gc;
                    if (gr < cur.d->rows) {
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (gc + e < cur.d->cols) ptr[e] = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
                    }
                }
            }
        }
        if (!has_next) break;
        cur = nxt;
        local = nlocal;
    }
}

// ----------------------------------------------------------------- launch

constexpr int kMaxDevices = 64;

template <int T, int RB, Storage ST, Operand OP>
hipError_t launch_one(const KernelArgs& args, hipStream_t stream)
{
    constexpr int WT = (T / 32) / RB;
    constexpr int TPW = 4 / WT;
    static std::atomic<int> resident[kMaxDevices];  // workgroups that fit at once, per device
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    int cap = resident[dev].load(std::memory_order_relaxed);
    if (cap == 0) {
        int per_cu = 0, cus = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, ns_tiled_kernel<T, RB, ST, OP>, kThreads, 0);
        if (e != hipSuccess) return e;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        cap = (per_cu < 1 ? 1 : per_cu) * (cus < 1 ? 1 : cus);
        resident[dev].store(cap, std::memory_order_relaxed);
    }
    const int64_t n = args.tile_end - args.tile_begin;
    if (n <= 0) return hipSuccess;
    const int64_t groups = (n + TPW - 1) / TPW;
    const int grid = (int)(groups < cap ? groups : cap);
    hipLaunchKernelGGL((ns_tiled_kernel<T, RB, ST, OP>), dim3(grid), dim3(kThreads), 0, stream, args);
    return hipGetLastError();
}

template <int T, int RB, int CMODE>
hipError_t launch_f16(const KernelArgs& args, hipStream_t stream)
{
    constexpr int TPW = 4 / ((T / 32) / RB);
    static std::atomic<int> resident[kMaxDevices];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    int cap = resident[dev].load(std::memory_order_relaxed);
    if (cap == 0) {
        int per_cu = 0, cus = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, ns_tiled_f16_kernel<T, RB, CMODE>, kThreads, 0);
        if (e != hipSuccess) return e;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        cap = (per_cu < 1 ? 1 : per_cu) * (cus < 1 ? 1 : cus);
        resident[dev].store(cap, std::memory_order_relaxed);
    }
    const int64_t n = args.tile_end - args.tile_begin;
    if (n <= 0) return hipSuccess;
    const int64_t groups = (n + TPW - 1) / TPW;
    const int grid = (int)(groups < cap ? groups : cap);
    hipLaunchKernelGGL((ns_tiled_f16_kernel<T, RB, CMODE>), dim3(grid), dim3(kThreads), 0, stream, args);
    return hipGetLastError();
}

// Kernel choice per tile size: rows of a T <= 64 tile stay in one wave (no
// workgroup barriers); a T = 128 tile is split over four waves.
template <Storage ST, Operand OP>
hipError_t launch_T(int T, const KernelArgs& args, hipStream_t stream)
{
    switch (T) {
    case 32: return launch_one<32, 1, ST, OP>(args, stream);
    case 64: return launch_one<64, 2, ST, OP>(args, stream);
    case 128: return launch_one<128, 1, ST, OP>(args, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool has_kernel(int T, Storage st, Operand op)
{
    const bool t_ok = T == 32 || T == 64 || T == 128;
    if (!t_ok) return false;
    if (st == Storage::F32) return op == Operand::F32;
    return op == Operand::F16 || op == Operand::BF16;
}

hipError_t launch_ns_tiled(int T, Storage st, Operand op, const KernelArgs& args, hipStream_t stream)
{
    if (!has_kernel(T, st, op)) return hipErrorInvalidValue;
    if (st == Storage::F32) return launch_T<Storage::F32, Operand::F32>(T, args, stream);
    if (op == Operand::F16) {
        const int cm = args.c > 0.f ? 0 : (args.c < 0.f ? 1 : 2);
        switch (T * 4 + cm) {
        case 32 * 4 + 0: return launch_f16<32, 1, 0>(args, stream);
        case 32 * 4 + 1: return launch_f16<32, 1, 1>(args, stream);
        case 32 * 4 + 2: return launch_f16<32, 1, 2>(args, stream);
        case 64 * 4 + 0: return launch_f16<64, 2, 0>(args, stream);
        case 64 * 4 + 1: return launch_f16<64, 2, 1>(args, stream);
        case 64 * 4 + 2: return launch_f16<64, 2, 2>(args, stream);
        case 128 * 4 + 0: return launch_f16<128, 1, 0>(args, stream);
        case 128 * 4 + 1: return launch_f16<128, 1, 1>(args, stream);
        case 128 * 4 + 2: return launch_f16<128, 1, 2>(args, stream);
        default: return hipErrorInvalidValue;
        }
    }
    return launch_T<Storage::BF16, Operand::BF16>(T, args, stream);
}

}  // namespace himuon
