// Fused tiled Newton–Schulz kernels for rectangular Th x Tw tiles (gfx950).
//
// The tiling operator with Th x Tw blocks (Sec. 2.1; the tile-shape study of
// Sec. 6.3 runs such tiles through its fused kernel when Th Tw <= 16384): each
// tile goes through Phi_K (Sec. 2.2, eqs. ns_iteration / phi_k_def), iterated
// on its wide orientation. A wide tile (Th <= Tw) is the iterate X itself,
// M = Th rows by N = Tw columns; a tall tile (Th > Tw) is iterated as its
// transpose (Phi_K(S) = Phi_K(S^T)^T, the orientation rule), so that the Gram
// matrix A = X X^T is always the small M x M one.
//
// One workgroup of W waves owns a tile, for all K steps; wave w owns a
// column slab of X (all M rows, N/W columns) as fp32 row pieces (the layout
// of ns_tiled_kernels.hip: lane l holds row l % 32 and columns
// 8g + 4(l/32) + e of each 32 x 32 block). Per step:
//   - each wave forms the partial Gram X_w X_w^T of its slab from its own row
//     pieces (no data from other waves);
//   - the partials are summed through LDS in a fixed wave order, so every
//     wave holds the same fp32 A;
//   - every wave forms B = bA + cA^2 (M x M, small) and its slab of
//     aX + BX, the column pieces of its own slab coming from LDS (written by
//     the same wave, in its own region).
// The only cross-wave traffic is the M x M partials and their sum. Operands are rounded
// once to fp16/bf16 (round to nearest even) or stay fp32; accumulation and
// the epilogues are fp32 with an fp32 master iterate, as in the square
// generic kernel.
#include "ns_device.h"

#include <atomic>

namespace himuon {
namespace {

using namespace dev;

template <int N> struct RectShape {
    static constexpr int W = N / 32 >= 4 ? 4 : N / 32;  // waves per tile
    static constexpr int NBC = N / 32 / W;              // 32-column blocks per wave slab
};

template <int M, int N, Storage ST, Operand OP, bool TALL>
__global__ void __launch_bounds__(RectShape<N>::W * 64) ns_rect_kernel(const KernelArgs args)
{
    constexpr int W = RectShape<N>::W;
    constexpr int NBC = RectShape<N>::NBC;
    constexpr int NBR = M / 32;
    constexpr int S = OperandTraits<OP>::kSlots;
    constexpr int NC = OperandTraits<OP>::kChains;
    constexpr int TH = TALL ? N : M, TW = TALL ? M : N;  // the tile in the matrix's orientation
    static_assert(M % 32 == 0 && N % (32 * W) == 0 && M <= N, "rectangular tile shape");
    // LDS: one region per wave, used first for the wave's partial Gram (NBR^2
    // fp32 blocks) and then for the column pieces of its slab.
    constexpr int PART = NBR * NBR * 16 * 64;        // floats
    constexpr int XC = NBR * NBC * S * 64;           // 16-byte slots
    constexpr int REGION = PART * 4 > XC * 16 ? PART * 4 : XC * 16;  // bytes
    constexpr int NV = NBR * NBR * 4;                // 16-byte vectors of the Gram per lane
    __shared__ __attribute__((aligned(16))) unsigned char s_reg[W * REGION];
    __shared__ f32x4 s_total[NV * 64];               // the summed Gram
    __shared__ float s_red[2][W];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int li = lane & 31, lh = lane >> 5;
    const int t4 = li & 3, quad = li >> 2;
    const int xg = quad >> 1, xh = quad & 1;
    f32x4* const part4 = reinterpret_cast<f32x4*>(s_reg + wave * REGION);
    f32x4* const total4 = s_total;
    u32x4* const xc = reinterpret_cast<u32x4*>(s_reg + wave * REGION);
    const int slab0 = wave * NBC * 32;  // first iterate column of the wave's slab

    // Tall tiles: a row-major copy of the TH x TW tile in the storage type,
    // over the wave regions (they are free outside the K loop).
    constexpr int ES = ST == Storage::BF16 ? 2 : 4;  // bytes per element
    constexpr int EPC = 16 / ES;                      // elements per 16-byte chunk
    constexpr int CPR = TW / EPC;                     // chunks per tile row
    static_assert(!TALL || TH * TW * ES <= W * REGION, "a tall tile's copy fits the wave regions");
    auto stage_rows = [&](const void* base, int64_t ld, int64_t rows, int64_t cols, int64_t r0, int64_t c0,
                          bool vec) {
        for (int ch = threadIdx.x; ch < TH * CPR; ch += W * 64) {
            const int r = ch / CPR, cc = ch % CPR;
            const int64_t gr = r0 + r, gc = c0 + cc * EPC;
            u32x4 v;
            if (vec) {
                v = *(const gbl_u32x4*)(static_cast<const unsigned char*>(base) + (gr * ld + gc) * ES);
            } else {
                uint32_t h[4] = {0u, 0u, 0u, 0u};
                if constexpr (ST == Storage::BF16) {
                    const uint16_t* p = static_cast<const uint16_t*>(base) + gr * ld + gc;
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (gr < rows && gc + e < cols) h[e >> 1] |= (uint32_t)p[e] << (16 * (e & 1));
                } else {
                    const uint32_t* p = static_cast<const uint32_t*>(base) + gr * ld + gc;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (gr < rows && gc + e < cols) h[e] = p[e];
                }
                v = u32x4{h[0], h[1], h[2], h[3]};
            }
            *reinterpret_cast<u32x4*>(s_reg + (r * TW + cc * EPC) * ES) = v;
        }
    };
    auto unstage_rows = [&](void* base, int64_t ld, int64_t rows, int64_t cols, int64_t r0, int64_t c0, bool vec) {
        for (int ch = threadIdx.x; ch < TH * CPR; ch += W * 64) {
            const int r = ch / CPR, cc = ch % CPR;
            const int64_t gr = r0 + r, gc = c0 + cc * EPC;
            const u32x4 v = *reinterpret_cast<const u32x4*>(s_reg + (r * TW + cc * EPC) * ES);
            if (vec) {
                *(gbl_u32x4*)(static_cast<unsigned char*>(base) + (gr * ld + gc) * ES) = v;
            } else if (gr < rows) {
                if constexpr (ST == Storage::BF16) {
                    uint16_t* p = static_cast<uint16_t*>(base) + gr * ld + gc;
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (gc + e < cols) p[e] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
                } else {
                    uint32_t* p = static_cast<uint32_t*>(base) + gr * ld + gc;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (gc + e < cols) p[e] = v[e];
                }
            }
        }
    };
    // element (r, c) of the copy (tile row r, column c), widened to fp32, and its store
    auto stage_get = [&](int r, int c) -> float {
        if constexpr (ST == Storage::BF16)
            return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(s_reg)[r * TW + c] << 16);
        else
            return reinterpret_cast<const float*>(s_reg)[r * TW + c];
    };
    auto stage_put = [&](int r, int c, float v) {
        if constexpr (ST == Storage::BF16)
            reinterpret_cast<uint16_t*>(s_reg)[r * TW + c] = (uint16_t)(pack2<Operand::BF16>(v, 0.f) & 0xffffu);
        else
            reinterpret_cast<float*>(s_reg)[r * TW + c] = v;
    };

    const int64_t n_tiles = args.tile_end - args.tile_begin;
    int mhint = 0;
    for (int64_t local = blockIdx.x; local < n_tiles; local += gridDim.x) {
        const int64_t tile = args.tile_begin + local;
        mhint = find_matrix_from(args, tile, mhint);
        const ConstDesc& d = desc_table(args)[mhint];
        const uint32_t lt = (uint32_t)(tile - d.tile_begin);
        const uint32_t tc = (uint32_t)d.tiles_c;
        const uint32_t tr = lt / tc;
        const int64_t row0 = (int64_t)tr * TH, col0 = (int64_t)(lt - tr * tc) * TW;
        const bool full = row0 + TH <= d.rows && col0 + TW <= d.cols;
        const bool vin = !TALL && full && (d.flags & MAT_VEC_IN);
        const bool vout = !TALL && full && (d.flags & MAT_VEC_OUT);

        // ---- gather the wave's slab of the iterate (zero padded) as fp32 row pieces.
        //      A tall tile goes through LDS: the workgroup moves its rows in
        //      16-byte chunks into a row-major copy, and each wave reads the
        //      columns of that copy as the rows of X = S^T.
        f32x16 X[NBR][NBC];
        if constexpr (TALL) {
            const bool vin_t = full && (d.flags & MAT_VEC_IN);
            stage_rows(d.in, d.ld_in, d.rows, d.cols, row0, col0, vin_t);
            __syncthreads();
#pragma unroll
            for (int I = 0; I < NBR; ++I)
#pragma unroll
                for (int q = 0; q < NBC; ++q)
#pragma unroll
                    for (int g = 0; g < 4; ++g)
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            X[I][q][4 * g + e] = stage_get(slab0 + 32 * q + 8 * g + 4 * lh + e, 32 * I + li);
            __syncthreads();  // the K loop reuses the staging area
        } else {
#pragma unroll
            for (int I = 0; I < NBR; ++I)
#pragma unroll
                for (int q = 0; q < NBC; ++q)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int64_t i = 32 * I + li, j = slab0 + 32 * q + 8 * g + 4 * lh;
                        const f32x4 v = load4<ST>(d.in, row0 + i, col0 + j, d.ld_in, d.rows, d.cols, vin);
#pragma unroll
                        for (int e = 0; e < 4; ++e) X[I][q][4 * g + e] = v[e];
                    }
        }

        // ---- X_0 = S / ||S||_F after an exact power-of-two pre-scale (the
        //      fp32 sum of squares neither overflows nor underflows)
        float mx = 0.f;
#pragma unroll
        for (int I = 0; I < NBR; ++I)
#pragma unroll
            for (int q = 0; q < NBC; ++q)
#pragma unroll
                for (int v = 0; v < 16; ++v) mx = fmaxf(mx, fabsf(X[I][q][v]));
        mx = wave_max(mx);
        if (lane == 0) s_red[0][wave] = mx;
        __syncthreads();
        mx = s_red[0][0];
#pragma unroll
        for (int w = 1; w < W; ++w) mx = fmaxf(mx, s_red[0][w]);
        int ex = 0;
        (void)frexpf(mx, &ex);
        const float s1 = ldexpf(1.f, -(ex / 2)), s2 = ldexpf(1.f, -(ex - ex / 2));
        float ss = 0.f;
#pragma unroll
        for (int I = 0; I < NBR; ++I)
#pragma unroll
            for (int q = 0; q < NBC; ++q)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const float y = X[I][q][v] * s1 * s2;
                    X[I][q][v] = y;
                    ss = fmaf(y, y, ss);
                }
        ss = wave_sum(ss);
        if (lane == 0) s_red[1][wave] = ss;
        __syncthreads();
        ss = s_red[1][0];
#pragma unroll
        for (int w = 1; w < W; ++w) ss += s_red[1][w];
        // fp32 operands: the exact power-of-two normalisation (exact_norm)
        float inv = ss > 0.f ? 1.f / sqrtf(ss) : 0.f;  // Phi_K(0) = 0
        ExactNorm en{};
        if constexpr (OP == Operand::F32) {
            en = exact_norm(ss, args.b, args.c);
            inv = en.scale;
        }
#pragma unroll
        for (int I = 0; I < NBR; ++I)
#pragma unroll
            for (int q = 0; q < NBC; ++q) X[I][q] *= inv;

        // ---- K Newton–Schulz steps, all on chip
        for (int k = 0; k < args.K; ++k) {
            u32x4 Xop[NBR][NBC][S];
#pragma unroll
            for (int I = 0; I < NBR; ++I)
#pragma unroll
                for (int q = 0; q < NBC; ++q)
#pragma unroll
                    for (int s = 0; s < S; ++s) Xop[I][q][s] = make_slot<OP>(X[I][q], s);

            // partial Gram of the slab: block (I, J) as row pieces of rows I
            f32x16 G[NBR][NBR];
            {
                f32x16 Gc[NBR][NBR][NC];
#pragma unroll
                for (int I = 0; I < NBR; ++I)
#pragma unroll
                    for (int J = 0; J < NBR; ++J)
#pragma unroll
                        for (int ch = 0; ch < NC; ++ch) Gc[I][J][ch] = f32x16{};
#pragma unroll
                for (int q = 0; q < NBC; ++q)
#pragma unroll
                    for (int s = 0; s < S; ++s)
#pragma unroll
                        for (int J = 0; J < NBR; ++J)
#pragma unroll
                            for (int I = 0; I < NBR; ++I) mma<OP>(Xop[J][q][s], Xop[I][q][s], Gc[I][J]);
#pragma unroll
                for (int I = 0; I < NBR; ++I)
#pragma unroll
                    for (int J = 0; J < NBR; ++J) G[I][J] = chain_sum<NC>(Gc[I][J]);
            }

            // sum of the partials. Wave w sums the 16-byte vectors v = w, w + W, ...
            // of the partials in wave order 0 .. W-1 and stores them to the
            // total; every wave then reads the whole total, so all hold the
            // same fp32 A. A wave's region holds only its own column pieces
            // between the last barrier of a step and here, so it overwrites
            // them without waiting for the others.
#pragma unroll
            for (int I = 0; I < NBR; ++I)
#pragma unroll
                for (int J = 0; J < NBR; ++J)
#pragma unroll
                    for (int v4 = 0; v4 < 4; ++v4)
                        part4[((I * NBR + J) * 4 + v4) * 64 + lane] =
                            f32x4{G[I][J][4 * v4], G[I][J][4 * v4 + 1], G[I][J][4 * v4 + 2], G[I][J][4 * v4 + 3]};
            __syncthreads();
#pragma unroll
            for (int vi = 0; vi < NV; vi += W) {
                if (vi + wave < NV) {
                    const int idx = (vi + wave) * 64 + lane;
                    f32x4 acc = reinterpret_cast<const f32x4*>(s_reg)[idx];
#pragma unroll
                    for (int w = 1; w < W; ++w) acc += reinterpret_cast<const f32x4*>(s_reg + w * REGION)[idx];
                    total4[idx] = acc;
                }
            }
            __syncthreads();  // every partial is summed; every wave reads the total
#pragma unroll
            for (int I = 0; I < NBR; ++I)
#pragma unroll
                for (int J = 0; J < NBR; ++J)
#pragma unroll
                    for (int v4 = 0; v4 < 4; ++v4) {
                        const f32x4 t = total4[((I * NBR + J) * 4 + v4) * 64 + lane];
#pragma unroll
                        for (int e = 0; e < 4; ++e) G[I][J][4 * v4 + e] = t[e];
                    }

            // column pieces of the slab for the B X product (own region)
#pragma unroll
            for (int Kb = 0; Kb < NBR; ++Kb)
#pragma unroll
                for (int q = 0; q < NBC; ++q)
#pragma unroll
                    for (int gp = 0; gp < 4; ++gp) {
                        const int lane_dst = xh * 32 + 8 * gp + 4 * lh + t4;
                        if constexpr (OP == Operand::F32) {
                            const f32x4 c = {X[Kb][q][4 * gp + 0], X[Kb][q][4 * gp + 1], X[Kb][q][4 * gp + 2],
                                             X[Kb][q][4 * gp + 3]};
                            const f32x4 o = quad_transpose32(c, t4);
                            xc[((Kb * NBC + q) * S + xg) * 64 + lane_dst] = __builtin_bit_cast(u32x4, o);
                        } else {
                            const u32x4& w = Xop[Kb][q][gp >> 1];
                            const u32x2 o = quad_transpose16(w[(gp & 1) * 2], w[(gp & 1) * 2 + 1], t4);
                            u32x2* dst = reinterpret_cast<u32x2*>(&xc[((Kb * NBC + q) * S + (xg >> 1)) * 64 + lane_dst]);
                            dst[xg & 1] = o;
                        }
                    }

            // B = bA + cA^2 (16-bit operands: accumulated in place as
            // c((b/c)A + A A^T); fp32: A^2 in zero-started chains, then one
            // fused b A + c A^2)
            if (args.c != 0.f) {
                u32x4 Aop[NBR][NBR][S];
#pragma unroll
                for (int I = 0; I < NBR; ++I)
#pragma unroll
                    for (int J = 0; J < NBR; ++J) {
#pragma unroll
                        for (int s = 0; s < S; ++s) Aop[I][J][s] = make_slot<OP>(G[I][J], s);
                        if constexpr (OP != Operand::F32) G[I][J] *= args.b_over_c;
                    }
                f32x16 Gc[NBR][NBR][NC];
#pragma unroll
                for (int I = 0; I < NBR; ++I)
#pragma unroll
                    for (int J = 0; J < NBR; ++J) {
                        if constexpr (OP == Operand::F32) Gc[I][J][0] = f32x16{};
                        else Gc[I][J][0] = G[I][J];
#pragma unroll
                        for (int ch = 1; ch < NC; ++ch) Gc[I][J][ch] = f32x16{};
                    }
#pragma unroll
                for (int Jk = 0; Jk < NBR; ++Jk)
#pragma unroll
                    for (int s = 0; s < S; ++s)
#pragma unroll
                        for (int J = 0; J < NBR; ++J)
#pragma unroll
                            for (int I = 0; I < NBR; ++I) mma<OP>(Aop[J][Jk][s], Aop[I][Jk][s], Gc[I][J]);
#pragma unroll
                for (int I = 0; I < NBR; ++I)
#pragma unroll
                    for (int J = 0; J < NBR; ++J) {
                        const f32x16 sq = chain_sum<NC>(Gc[I][J]);
                        if constexpr (OP == Operand::F32) {
#pragma unroll
                            for (int v = 0; v < 16; ++v) G[I][J][v] = poly2(en, G[I][J][v], sq[v]);
                        } else {
                            G[I][J] = sq * args.c;
                        }
                    }
            } else {
#pragma unroll
                for (int I = 0; I < NBR; ++I)
#pragma unroll
                    for (int J = 0; J < NBR; ++J) {
                        if constexpr (OP == Operand::F32) {
#pragma unroll
                            for (int v = 0; v < 16; ++v) G[I][J][v] = fmaf(en.bh, G[I][J][v], en.bl * G[I][J][v]);
                        } else {
                            G[I][J] *= args.b;
                        }
                    }
            }

            // X <- aX + B X on the slab
            u32x4 Bop[NBR][NBR][S];
#pragma unroll
            for (int I = 0; I < NBR; ++I)
#pragma unroll
                for (int Kb = 0; Kb < NBR; ++Kb)
#pragma unroll
                    for (int s = 0; s < S; ++s) Bop[I][Kb][s] = make_slot<OP>(G[I][Kb], s);
            {
                f32x16 Pc[NBR][NBC][NC];
#pragma unroll
                for (int I = 0; I < NBR; ++I)
#pragma unroll
                    for (int q = 0; q < NBC; ++q) {
                        if constexpr (OP == Operand::F32) Pc[I][q][0] = f32x16{};
                        else Pc[I][q][0] = X[I][q] * args.a;
#pragma unroll
                        for (int ch = 1; ch < NC; ++ch) Pc[I][q][ch] = f32x16{};
                    }
#pragma unroll
                for (int q = 0; q < NBC; ++q)
#pragma unroll
                    for (int Kb = 0; Kb < NBR; ++Kb)
#pragma unroll
                        for (int s = 0; s < S; ++s) {
                            const u32x4 opa = xc[((Kb * NBC + q) * S + s) * 64 + lane];
#pragma unroll
                            for (int I = 0; I < NBR; ++I) mma<OP>(opa, Bop[I][Kb][s], Pc[I][q]);
                        }
#pragma unroll
                for (int I = 0; I < NBR; ++I)
#pragma unroll
                    for (int q = 0; q < NBC; ++q) {
                        const f32x16 bx = chain_sum<NC>(Pc[I][q]);
                        if constexpr (OP == Operand::F32) {
#pragma unroll
                            for (int v = 0; v < 16; ++v) X[I][q][v] = fmaf(args.a, X[I][q][v], bx[v]);
                        } else {
                            X[I][q] = bx;
                        }
                    }
            }
        }

        // ---- write back the unpadded part (a tall tile through the LDS copy)
        if constexpr (OP == Operand::F32) {
#pragma unroll
            for (int I = 0; I < NBR; ++I)
#pragma unroll
                for (int q = 0; q < NBC; ++q) X[I][q] *= en.out;
        }
        if constexpr (TALL) {
            __syncthreads();  // every wave is done with its region of the staging area
#pragma unroll
            for (int I = 0; I < NBR; ++I)
#pragma unroll
                for (int q = 0; q < NBC; ++q)
#pragma unroll
                    for (int g = 0; g < 4; ++g)
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            stage_put(slab0 + 32 * q + 8 * g + 4 * lh + e, 32 * I + li, X[I][q][4 * g + e]);
            __syncthreads();
            const bool vout_t = full && (d.flags & MAT_VEC_OUT);
            unstage_rows(d.out, d.ld_out, d.rows, d.cols, row0, col0, vout_t);
        } else {
#pragma unroll
            for (int I = 0; I < NBR; ++I)
#pragma unroll
                for (int q = 0; q < NBC; ++q)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int64_t i = 32 * I + li, j = slab0 + 32 * q + 8 * g + 4 * lh;
                        const f32x4 v = {X[I][q][4 * g + 0], X[I][q][4 * g + 1], X[I][q][4 * g + 2],
                                         X[I][q][4 * g + 3]};
                        store4<ST>(d.out, row0 + i, col0 + j, d.ld_out, d.rows, d.cols, vout, v);
                    }
        }
        __syncthreads();  // the next tile's normalisation reuses s_red (and a tall tile's staging area)
    }
}

constexpr int kMaxDevices = 64;

template <int M, int N, Storage ST, Operand OP, bool TALL>
hipError_t launch_rect(const KernelArgs& args, hipStream_t stream)
{
    constexpr int threads = RectShape<N>::W * 64;
    static std::atomic<int> resident[kMaxDevices];  // workgroups that fit at once, per device
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    int cap = resident[dev].load(std::memory_order_relaxed);
    if (cap == 0) {
        int per_cu = 0, cus = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, ns_rect_kernel<M, N, ST, OP, TALL>, threads, 0);
        if (e != hipSuccess) return e;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        cap = (per_cu < 1 ? 1 : per_cu) * (cus < 1 ? 1 : cus);
        resident[dev].store(cap, std::memory_order_relaxed);
    }
    const int64_t n = args.tile_end - args.tile_begin;
    if (n <= 0) return hipSuccess;
    const int grid = (int)(n < cap ? n : cap);
    hipLaunchKernelGGL((ns_rect_kernel<M, N, ST, OP, TALL>), dim3(grid), dim3(threads), 0, stream, args);
    return hipGetLastError();
}

template <Storage ST, Operand OP, bool TALL>
hipError_t launch_shape(int m, int n, const KernelArgs& args, hipStream_t stream)
{
    switch (m * 4096 + n) {
    case 32 * 4096 + 64: return launch_rect<32, 64, ST, OP, TALL>(args, stream);
    case 32 * 4096 + 128: return launch_rect<32, 128, ST, OP, TALL>(args, stream);
    case 32 * 4096 + 256: return launch_rect<32, 256, ST, OP, TALL>(args, stream);
    default: break;
    }
    // (fp32 operands keep four accumulator chains per output block: at
    // M = 64, or N = 512, a wave's chains alone fill the register file and
    // spill; those shapes run on the library GEMMs)
    if constexpr (OP != Operand::F32) {
        switch (m * 4096 + n) {
        case 32 * 4096 + 512: return launch_rect<32, 512, ST, OP, TALL>(args, stream);
        case 64 * 4096 + 128: return launch_rect<64, 128, ST, OP, TALL>(args, stream);
        case 64 * 4096 + 256: return launch_rect<64, 256, ST, OP, TALL>(args, stream);
        default: break;
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool has_rect_kernel(int Th, int Tw, Storage st, Operand op)
{
    const int m = Th < Tw ? Th : Tw, n = Th < Tw ? Tw : Th;
    const bool small = m == 32 && (n == 64 || n == 128 || n == 256);
    const bool large = (m == 32 && n == 512) || (m == 64 && (n == 128 || n == 256));
    if (st == Storage::F32) return op == Operand::F32 && small;
    return (op == Operand::F16 || op == Operand::BF16) && (small || large);
}

hipError_t launch_ns_rect(int Th, int Tw, Storage st, Operand op, const KernelArgs& args, hipStream_t stream)
{
    if (!has_rect_kernel(Th, Tw, st, op)) return hipErrorInvalidValue;
    const bool tall = Th > Tw;
    const int m = tall ? Tw : Th, n = tall ? Th : Tw;
    if (st == Storage::F32)
        return tall ? launch_shape<Storage::F32, Operand::F32, true>(m, n, args, stream)
                    : launch_shape<Storage::F32, Operand::F32, false>(m, n, args, stream);
    if (op == Operand::F16)
        return tall ? launch_shape<Storage::BF16, Operand::F16, true>(m, n, args, stream)
                    : launch_shape<Storage::BF16, Operand::F16, false>(m, n, args, stream);
    return tall ? launch_shape<Storage::BF16, Operand::BF16, true>(m, n, args, stream)
                : launch_shape<Storage::BF16, Operand::BF16, false>(m, n, args, stream);
}

}  // namespace himuon
