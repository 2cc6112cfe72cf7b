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
#include "ns_device.h"

#include <atomic>

namespace himuon {
namespace {

using namespace dev;

constexpr int kThreads = 256;  // four waves per workgroup

// T: tile size; RB: 32-row blocks per wave. A tile is spread over
// WT = T/(32 RB) waves, and a workgroup of four waves runs 4/WT tiles.
// OPT: the optimizer step of Alg. 1 rides on the tile I/O (KernelArgs): the
// gather loads G and M, stores M <- beta M + G and takes the lookahead
// G + beta M (Nesterov) or M, formed from the stored M, as the tile; the
// write-back loads W and stores (1 - lr lambda) W - lr tau U.
template <int T, int RB, Storage ST, Operand OP, bool OPT = false>
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

    int mhint = 0;  // owner of the wave's previous valid tile
    for (int64_t grp = blockIdx.x; grp < n_groups; grp += gridDim.x) {
        const int64_t local = grp * TPW + tslot;
        const bool valid = local < n_tiles;
        if constexpr (!SHARED_ROWS || TPW == 1) {
            if (!valid) continue;  // no workgroup barrier depends on this wave
        }
        const int64_t tile = args.tile_begin + (valid ? local : 0);

        // matrix owning the tile: last descriptor with tile_begin <= tile.
        // A wave's valid tiles only grow, so the search starts from the
        // previous owner; an idle wave (the chunk's first tile) searches all.
        const ConstDesc* const descs = desc_table(args);
        int lo;
        if (valid) {
            mhint = find_matrix_from(args, tile, mhint);
            lo = mhint;
        } else {
            int l = 0, hi = args.n_mats - 1;
            while (l < hi) {
                const int mid = (l + hi + 1) >> 1;
                if (descs[mid].tile_begin <= tile) l = mid;
                else hi = mid - 1;
            }
            lo = __builtin_amdgcn_readfirstlane(l);
        }
        const ConstDesc& d = descs[lo];
        // (32-bit: tile ids of one call fit in 32 bits, checked on the host)
        const uint32_t lt = (uint32_t)(tile - d.tile_begin);
        const uint32_t tc = (uint32_t)d.tiles_c;
        const uint32_t tr = lt / tc;
        const int64_t row0 = (int64_t)tr * T, col0 = (int64_t)(lt - tr * tc) * T;
        const bool full = row0 + T <= d.rows && col0 + T <= d.cols;
        const bool vin = full && (d.flags & MAT_VEC_IN);
        const bool vout = full && (d.flags & MAT_VEC_OUT);
        const int64_t rows_eff = valid ? d.rows : 0;  // an idle wave reads zeros

        void* mom = nullptr;
        float tau = 0.f;
        if constexpr (OPT) {
            const ConstOpt& O = opt_table(args)[lo];
            mom = O.mom;
            tau = O.tau;
        }

        // ---- gather the tile (zero padded) into fp32 row pieces
        f32x16 X[RB][NB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int64_t gr = row0 + 32 * (p0 + rb) + li;
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int64_t gc = col0 + 32 * q + 8 * g + 4 * lh;
                    const f32x4 v = load4<ST>(d.in, gr, gc, d.ld_in, rows_eff, d.cols, vin);
                    float x4[4] = {v[0], v[1], v[2], v[3]};
                    if constexpr (OPT) {
                        // (the momentum shares the gradient's layout; padding stays zero)
                        const f32x4 m = load4<ST>(mom, gr, gc, d.ld_in, rows_eff, d.cols, vin);
                        const f32x4 mn = stored4<ST>(f32x4{args.beta * m[0] + x4[0], args.beta * m[1] + x4[1],
                                                           args.beta * m[2] + x4[2], args.beta * m[3] + x4[3]});
                        if (valid) store4<ST>(mom, gr, gc, d.ld_in, d.rows, d.cols, vin, mn);
                        const float nb = args.nesterov ? args.beta : 0.f;
                        const float keep = args.nesterov ? 1.f : 0.f;
                        const float mb = args.nesterov ? 0.f : 1.f;
#pragma unroll
                        for (int e = 0; e < 4; ++e) x4[e] = keep * x4[e] + nb * mn[e] + mb * mn[e];
                    }
                    X[rb][q][4 * g + 0] = x4[0];
                    X[rb][q][4 * g + 1] = x4[1];
                    X[rb][q][4 * g + 2] = x4[2];
                    X[rb][q][4 * g + 3] = x4[3];
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
        // 16-bit operands round the tile anyway: X_0 = S / ||S||_F. fp32
        // operands: the exact power-of-two normalisation (exact_norm), the
        // rest of ||S||_F in the step's coefficients and the output factor.
        float inv = ss > 0.f ? 1.f / sqrtf(ss) : 0.f;  // Phi_K(0) = 0
        ExactNorm en{};
        if constexpr (OP == Operand::F32) {
            en = exact_norm(ss, args.b, args.c);
            inv = en.scale;
        }
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
                            for (int v = 0; v < 16; ++v) G[rb][J][v] = poly2(en, G[rb][J][v], sq[v]);
                        } else {
                            G[rb][J] = sq * args.c;
                        }
                    }
            } else {
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int J = 0; J < NB; ++J) {
                        if constexpr (OP == Operand::F32) {
#pragma unroll
                            for (int v = 0; v < 16; ++v) G[rb][J][v] = fmaf(en.bh, G[rb][J][v], en.bl * G[rb][J][v]);
                        } else {
                            G[rb][J] *= args.b;
                        }
                    }
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
        if constexpr (OP == Operand::F32) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int q = 0; q < NB; ++q) X[rb][q] *= en.out;
        }
        if (valid) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                const int64_t gr = row0 + 32 * (p0 + rb) + li;
#pragma unroll
                for (int q = 0; q < NB; ++q)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int64_t gc = col0 + 32 * q + 8 * g + 4 * lh;
                        f32x4 v = {X[rb][q][4 * g + 0], X[rb][q][4 * g + 1], X[rb][q][4 * g + 2],
                                   X[rb][q][4 * g + 3]};
                        if constexpr (OPT) {
                            // U as the storage type holds it, then the update of the loaded W
                            const f32x4 u = stored4<ST>(v);
                            const f32x4 w = load4<ST>(d.out, gr, gc, d.ld_out, d.rows, d.cols, vout);
                            const float step = args.lr * tau;
#pragma unroll
                            for (int e = 0; e < 4; ++e) v[e] = args.decay * w[e] - step * u[e];
                        }
                        store4<ST>(d.out, gr, gc, d.ld_out, d.rows, d.cols, vout, v);
                    }
            }
        }
    }
}

// ----------------------------------------------------------------- launch

constexpr int kMaxDevices = 64;

template <int T, int RB, Storage ST, Operand OP, bool OPT>
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
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, ns_tiled_kernel<T, RB, ST, OP, OPT>, kThreads, 0);
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
    hipLaunchKernelGGL((ns_tiled_kernel<T, RB, ST, OP, OPT>), dim3(grid), dim3(kThreads), 0, stream, args);
    return hipGetLastError();
}

// Kernel choice per tile size: rows of a T <= 64 tile stay in one wave (no
// workgroup barriers); a T = 128 tile is split over four waves.
template <Storage ST, Operand OP>
hipError_t launch_T(int T, const KernelArgs& args, hipStream_t stream)
{
    if (args.step) {
        switch (T) {
        case 32: return launch_one<32, 1, ST, OP, true>(args, stream);
        case 64: return launch_one<64, 2, ST, OP, true>(args, stream);
        case 128: return launch_one<128, 1, ST, OP, true>(args, stream);
        default: return hipErrorInvalidValue;
        }
    }
    switch (T) {
    case 32: return launch_one<32, 1, ST, OP, false>(args, stream);
    case 64: return launch_one<64, 2, ST, OP, false>(args, stream);
    case 128: return launch_one<128, 1, ST, OP, false>(args, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool has_kernel(int T, Storage st, Operand op)
{
    if (T == 256) return st == Storage::BF16 && op == Operand::F16;  // fp16-operand kernel only
    const bool t_ok = T == 32 || T == 64 || T == 128;
    if (!t_ok) return false;
    if (st == Storage::F32) return op == Operand::F32;
    return op == Operand::F16 || op == Operand::BF16;
}

hipError_t launch_ns_tiled(int T, Storage st, Operand op, const KernelArgs& args, hipStream_t stream)
{
    if (!has_kernel(T, st, op)) return hipErrorInvalidValue;
    if (st == Storage::F32) return launch_T<Storage::F32, Operand::F32>(T, args, stream);
    if (op == Operand::F16) return launch_ns_tiled_f16(T, args, stream);
    return launch_T<Storage::BF16, Operand::BF16>(T, args, stream);
}

}  // namespace himuon
