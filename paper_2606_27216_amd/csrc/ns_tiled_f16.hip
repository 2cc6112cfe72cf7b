// fp16-operand tiled Newton–Schulz kernel for gfx950 (MI355X), bf16 storage.
//
// Evaluates Phi_K (Sec. 2.2, eqs. ns_iteration / ns_quintic / phi_k_def) on
// every tile of a chunk of the batched tile set (Sec. 4.1, eq. tiled_ns;
// Sec. 4.4.2). Built with MFMA results kept in architectural VGPRs
// (-amdgpu-mfma-vgpr-form): every accumulator is converted by vector ALU
// instructions right after its product, and AGPR-resident accumulators
// would need a copy for each conversion.
#include "ns_device.h"

#include <atomic>
#include <type_traits>

namespace himuon {
namespace {

using namespace dev;

// ------------------------------------------------ fp16-operand kernel
//
// Same tile map, restructured so that no vector-ALU work but the fp16
// conversions is left in the K loop. The state is Z = X |c|^(1/4) (exact
// rescaling of the iterate), for which one step of eq. (ns_iteration) reads
//     Z <- (a I + sigma H^2 + b' H) Z,   H = Z Z^T,
// with b' = b / sqrt|c| and sigma = sign(c): the c-coefficient becomes +-1.
// Completing the square, with M = H + (sigma b' / 2) I,
//     a I + sigma H^2 + b' H = sigma M^2 + a' I,   a' = a - b^2 / (4c),
// so the Gram product, seeded with the shift on its diagonal blocks, yields M
// directly, the polynomial is the single product M M seeded with sigma a' I,
// and a step is three MFMA products with nothing between them but the fp16
// conversions of their results. Between steps the iterate is held as fp16
// operands only (near convergence a I + P has eigenvalues of order one, so
// rounding its product does not amplify). The normalisation multiplies by
// |c|^(1/4) and the store by |c|^(-1/4). c = 0 takes a I + b H.
//
// Z is shared through one row-major fp16 copy of the tile (see kRowStride).
// Gram operands of the other waves' rows are read from it as row pieces; the
// column operands of the third product come from it through
// ds_read_b64_tr_b16, which returns in every lane quad a 4x4 transpose of
// four rows supplied by the other lanes of its 16-lane group. A 128-tile
// computes only the upper blocks of the symmetric H and aI + P and shares
// them as 32x32 fp16 blocks (see ns_steps_sym); a 256-tile has no room for
// them and uses a regrouped step (see ns_steps_chain). Tiles of one wave
// need no sharing. A wave works on the blocks of its row in the rotated
// order J = (p + j) mod NB, so its own row blocks come from registers.
//
// Tiles are processed in rounds; the HBM loads of a wave's next tile are
// issued before the current tile is written back.

// Sum over the 64 lanes in a fixed order: butterflies inside each 16-lane
// row (quad swaps, half-row and row mirrors) leave every lane of a row with
// the row's sum; row broadcasts then add row 0 into row 1 and row 2 into row
// 3, and lane 31 into rows 2 and 3, so lane 63 holds (r2 + r3) + (r0 + r1).
// (DPP reads from lanes that exist only; rows a broadcast does not write get
// 0, the identity of the sum, so each step folds into one DPP add.)
template <int CTRL, int ROW_MASK> HM_DEV float dpp_add(float v)
{
    return v + __uint_as_float((uint32_t)__builtin_amdgcn_update_dpp(0, (int)__float_as_uint(v), CTRL, ROW_MASK, 0xF, false));
}

HM_DEV float wave_sum_f32(float v)
{
    v = dpp_add<0xB1, 0xF>(v);  // quad_perm [1, 0, 3, 2]
    v = dpp_add<0x4E, 0xF>(v);  // quad_perm [2, 3, 0, 1]
    v = dpp_add<0x141, 0xF>(v);  // row_half_mirror
    v = dpp_add<0x140, 0xF>(v);  // row_mirror
    v = dpp_add<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
    v = dpp_add<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
    return __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(v), 63));
}

HM_DEV uint32_t wave_max_u32(uint32_t v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o));
    return v;
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

// Row-major fp16 copy of Z. Bytes per row: an odd multiple of 64 (or 64
// past an even one), so that the row offset modulo the 256-byte bank space
// steps by a quarter (64 bytes) between consecutive rows. Within each 64-byte
// segment (32 columns) the 8-byte chunk c of row r sits at chunk
// c ^ rm_swz(r). On gfx950 (measured with the LDS bank-conflict counter):
// ds_read_b64 and ds_read_b64_tr_b16 serve 32 lanes per pass from 64 banks,
// ds_write_b64 16 consecutive lanes per pass from 32 banks (128 bytes), and
// ds_read_b128 16 lanes per pass, lanes {0-7, 24-31} and {8-15, 16-23} of
// each half wave together. A row-piece access touches one chunk of each of
// 32 consecutive rows: the row offset separates rows by r mod 4 (reads) or
// r mod 2 (writes), and the swizzle takes eight distinct values over the
// remaining row bits of each pass (bits 2-4 resp. 1-3), so both are
// conflict-free. A transposing read touches 8 chunks of 4 consecutive rows
// per pass, which the row offset alone separates.
HM_DEV int rm_swz(int r) { return ((r >> 1) & 7) ^ ((r >> 4) & 1); }

template <int T> constexpr int kRowStride = ((2 * T / 64) % 2 == 1) ? 2 * T : 2 * T + 64;

// Workgroup shape of the fp16 kernel. A tile split over WT > 1 waves is
// one workgroup of WT waves; tiles kept by one wave come four to a
// workgroup. A wave that owns two row blocks of a 128-tile keeps its state,
// accumulators and the next tile's prefetched rows in up to 512 registers
// (one wave per SIMD); everything else runs two waves per SIMD.
template <int T, int RB> struct F16Shape {
    static constexpr int NB = T / 32;
    static constexpr int WT = NB / RB;
    static constexpr int TPW = WT > 1 ? 1 : 4;
    static constexpr int kThreads = 64 * WT * TPW;
    static constexpr bool kWide = T == 128 && RB == 2;
    // a 256-tile: one per CU, four waves of two row blocks, chain-form step
    static constexpr bool kChain = T == 256;
    // a 128-tile evaluates only the upper blocks of the symmetric H and aI + P
    static constexpr bool kSym = kWide;
    static constexpr int kMinWavesPerEU = (kWide || kChain) ? 1 : 2;
    // next tile's loads issued before the K loop (registers permitting)
    static constexpr bool kEarlyPrefetch = kWide;
};

// CMODE: 0 for c > 0, 1 for c < 0, 2 for c = 0 (sign(c) and the c = 0
// shortcut are compile-time, so no branch of the K loop is if-converted).
// RB: 32-row blocks owned by one wave; a tile is spread over NB / RB waves.
// Every operand read from LDS feeds RB MFMAs.
// OPT: the optimizer step of Alg. 1 rides on the tile I/O (KernelArgs):
// the staging turns the loaded G and M into the stored new M and the
// lookahead, and the write-back turns U into the decayed, tau-scaled update
// of the loaded W. Without OPT the kernel is the map alone.
template <int T, int RB, int CMODE, bool OPT>
__global__ void __launch_bounds__((F16Shape<T, RB>::kThreads), (F16Shape<T, RB>::kMinWavesPerEU)) ns_tiled_f16_kernel(const KernelArgs args)
{
    constexpr Storage ST = Storage::BF16;
    constexpr Operand OP = Operand::F16;
    constexpr int NB = T / 32;      // row blocks per tile
    constexpr int WT = NB / RB;     // waves per tile
    static_assert(NB % RB == 0 && WT >= 1 && WT <= 4, "tile split");
    constexpr int TPW = F16Shape<T, RB>::TPW;  // tiles per workgroup
    constexpr bool EARLY = F16Shape<T, RB>::kEarlyPrefetch && !OPT;  // (a step holds G and M: no room)
    constexpr int S = 2;
    constexpr int MAT = NB * NB * S * 64;  // 16-byte slots of H
    constexpr bool SHARED = WT > 1;
    static_assert(!SHARED || TPW == 1, "a workgroup that shares a tile runs one tile");
    constexpr int NO = NB - RB;     // row blocks owned by the other waves of the tile
    constexpr int NOA = NO > 0 ? NO : 1;
    constexpr int RS = kRowStride<T>;
    constexpr int RM = T * RS;
    constexpr int IT = NB * S;      // k iterations of one product

    // H slots; for the symmetric 128-tile step, 18 blocks of 32x32 fp16 (12 of H, 6 of aI + P)
    // A 64-tile (one wave) evaluates only the upper blocks of H and aI + P
    // too; its lower off-diagonal blocks come back through two 32x32 fp16
    // blocks of LDS per tile (c != 0 only).
    constexpr bool SYM64 = T == 64 && RB == 2 && WT == 1 && CMODE != 2;
    constexpr int NSLOT = F16Shape<T, RB>::kSym ? 18 * 2048 / 16
                          : SYM64 ? TPW * 2 * 2048 / 16
                          : ((SHARED && !F16Shape<T, RB>::kChain) ? TPW * MAT : 1);
    __shared__ u32x4 s_slots[NSLOT];
    __shared__ __attribute__((aligned(16))) uint8_t s_rm[TPW * RM];
    __shared__ float s_red[6][SHARED ? WT : 1];  // 2 tile parities x 3 reductions

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int tslot = wave / WT, p0 = (wave % WT) * RB;
    const int li = lane & 31, lh = lane >> 5;
    u32x4* const slots = s_slots + (SHARED ? tslot * MAT : 0);
    uint8_t* const rm = s_rm + tslot * RM;
    // Row pieces: this lane's columns 32q + 8g + 4lh of row li of a block are
    // chunk 2g + lh of the block's segment q.
    int rp_off[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) rp_off[g] = li * RS + 8 * ((2 * g + lh) ^ rm_swz(li));
    // The staged input and the packed output use the swizzle with its lowest
    // bit cleared (chunk c at c ^ (rm_swz(r) & 6)), in which the two 8-byte
    // halves of every aligned 16-byte pair keep their order: whole 16-byte
    // row chunks then move between HBM and LDS with no exchange in
    // registers, at the price of two-way bank conflicts on the four
    // row-piece accesses of each end of a tile.
    int io_rp[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) io_rp[g] = li * RS + 8 * ((2 * g + lh) ^ (rm_swz(li) & 6));
    // Transposing reads: supplier lane 4q' + m of 16-lane group G addresses
    // row 16s + 4(G/2) + m (+ 8x) and logical chunk 4(G%2) + q' of a block
    // segment, for the k half s of the block.
    const int grp16 = lane >> 4;
    int tr_off[S][2];
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
        for (int x = 0; x < 2; ++x) {
            const int row = 16 * s + 8 * x + 4 * (grp16 >> 1) + ((lane & 15) >> 2);
            const int chunk = 4 * (grp16 & 1) + (lane & 3);
            tr_off[s][x] = row * RS + 8 * (chunk ^ rm_swz(row));
        }
    // A diagonal block holds row li's column 8g + 4lh + e in register 4g + e,
    // so the diagonal entry of this lane (if any) is register vdiag.
    const int vdiag = (lh == ((li >> 2) & 1)) ? 4 * (li >> 3) + (li & 3) : -1;
    // Diagonal blocks that seed accumulators: sigma a' I for the polynomial
    // product (sigma a I for c = 0), and the shift (sigma b' / 2) I that turns
    // a diagonal Gram block into the same block of M (zero for c = 0).
    f32x16 diag_a = {}, diag_m = {};
    {
        const float sa = CMODE == 2 ? args.a : args.am;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            diag_a[v] = v == vdiag ? (CMODE == 1 ? -sa : sa) : 0.f;
            diag_m[v] = (CMODE != 2 && v == vdiag) ? args.hshift : 0.f;
        }
    }
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
        const void* in;
        void* out;
        int64_t rows, cols, ld_in, ld_out;
        int64_t row0, col0;
        int32_t vin, vout;  // (not bool: a struct with bools is not split into registers)
        void* mom;  // OPT: the momentum buffer (layout of `in`) and tau
        float tau;
    };
    int mhint = 0;
    auto locate = [&](int64_t local, TileLoc& L) {
        const int64_t tile = args.tile_begin + local;
        mhint = find_matrix_from(args, tile, mhint);
        const ConstDesc& D = desc_table(args)[mhint];
        L.in = D.in;
        L.out = D.out;
        L.rows = D.rows;
        L.cols = D.cols;
        L.ld_in = D.ld_in;
        L.ld_out = D.ld_out;
        // (32-bit: a 64-bit division would expand to a long scalar sequence)
        const uint32_t lt = (uint32_t)(tile - D.tile_begin);
        const uint32_t tc = (uint32_t)D.tiles_c;
        const uint32_t tr = lt / tc;
        L.row0 = (int64_t)tr * T;
        L.col0 = (int64_t)(lt - tr * tc) * T;
        const bool full = L.row0 + T <= L.rows && L.col0 + T <= L.cols;
        const int32_t fl = D.flags;  // (read unconditionally: no dependent scalar load)
        L.vin = full & ((fl & MAT_VEC_IN) != 0);
        L.vout = full & ((fl & MAT_VEC_OUT) != 0);
        if constexpr (OPT) {
            const ConstOpt& O = opt_table(args)[mhint];
            L.mom = O.mom;
            L.tau = O.tau;
        } else {
            L.mom = nullptr;
            L.tau = 0.f;
        }
    };
    // HBM traffic in whole row segments: a lane moves 16 bytes (8 bf16), a
    // row takes LPR lanes and one wave instruction RPI rows. The wave's own
    // RB row blocks take NI instructions; the row pieces are then reshaped
    // through the wave's own rows of the row-major copy.
    constexpr int LPR = T / 8;
    constexpr int RPI = 64 / LPR;
    constexpr int NI = 32 * RB / RPI;
    const int io_row = lane / LPR, io_cc = lane % LPR;  // row within an instruction, 16-byte chunk
    // The tile loop is compiled once per wave index of a shared 128-tile
    // (w = 0, 1): the wave's row blocks, and with them every LDS offset in the
    // K loop, become compile-time constants folded into the LDS instructions.
    const int p0_rt = p0;
    auto tile_loop = [&](auto wtag) {
    constexpr int WSPEC = decltype(wtag)::value;  // -1: not specialised
    const int p0 = WSPEC >= 0 ? RB * WSPEC : p0_rt;
    u32x4 raw[NI];
    u32x4 rawm[OPT ? NI : 1];  // OPT: the momentum rows of the tile
    // the wave's rows of the tile in `base` (leading dimension ld), zero
    // outside the matrix
    auto load_rows = [&](const TileLoc& L, const void* base, int64_t ld, bool vec, u32x4 (&dst)[NI]) {
        const int64_t gr0 = L.row0 + 32 * p0 + io_row;
        const int64_t gc = L.col0 + 8 * io_cc;
        if (vec) {  // whole tile inside, 16-byte aligned: straight vector loads
            const gbl_u32x4* src = (const gbl_u32x4*)(static_cast<const uint16_t*>(base) + gr0 * ld + gc);
            const int64_t step = (int64_t)RPI * ld / 8;  // u32x4 per RPI rows
#pragma unroll
            for (int i = 0; i < NI; ++i) dst[i] = src[i * step];
        } else {
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                const int64_t gr = gr0 + RPI * i;
                const uint16_t* ptr = static_cast<const uint16_t*>(base) + gr * ld + gc;
                uint32_t h[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
                if (gr < L.rows) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (gc + e < L.cols) h[e] = ptr[e];
                }
                dst[i] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
            }
        }
    };
    auto issue_loads = [&](const TileLoc& L) {
        load_rows(L, L.in, L.ld_in, L.vin, raw);
        if constexpr (OPT) load_rows(L, L.mom, L.ld_in, L.vin, rawm);
    };
    // byte offset of the 16-byte chunk io_cc of tile row `row` in the staging
    // layout of the row-major copy (io_rp)
    auto io_lds = [&](int row) -> int {
        return row * RS + 64 * (io_cc >> 2) + 16 * ((io_cc & 3) ^ (rm_swz(row) >> 1));
    };
    // The symmetric 128-tile step keeps its Z copy in a layout of aligned
    // 16-byte operand pairs (described at ns_steps_sym); its tiles are
    // staged in that layout too: a 16-byte row chunk goes in as two 8-byte
    // halves, and row pieces move as whole pairs.
    constexpr bool PAIRS = F16Shape<T, RB>::kSym;
    auto tsw = [](int r) { return ((r >> 1) ^ (r >> 2) ^ (r >> 4)) & 3; };
    int rpB[S];
#pragma unroll
    for (int s = 0; s < S; ++s) rpB[s] = li * RS + 16 * ((2 * s + lh) ^ tsw(li));
    // byte offset of half h (columns 8 io_cc + 4h .. +3) of staging chunk io_cc of
    // `row` (the pair swizzle is a function of the row within its 32-row block)
    auto io_half = [&](int row, int h) -> int {
        const int jj = io_cc & 3;
        return row * RS + 64 * (io_cc >> 2) + 16 * ((2 * (jj >> 1) + h) ^ tsw(row & 31)) + 8 * (jj & 1);
    };

    // Whole row segments of the own rows to HBM (16-byte chunks read back from
    // the row-major copy into `outv`), inside the matrix only.
    auto put_rows = [&](const TileLoc& L, void* base, int64_t ld, bool vec, const u32x4 (&v)[NI]) {
        const int64_t gr0 = L.row0 + 32 * p0 + io_row;
        const int64_t gc = L.col0 + 8 * io_cc;
        if (vec) {
            gbl_u32x4* dst = (gbl_u32x4*)(static_cast<uint16_t*>(base) + gr0 * ld + gc);
            const int64_t step = (int64_t)RPI * ld / 8;
#pragma unroll
            for (int i = 0; i < NI; ++i) dst[i * step] = v[i];
        } else {
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                const int64_t gr = gr0 + RPI * i;
                uint16_t* ptr = static_cast<uint16_t*>(base) + gr * ld + gc;
                if (gr < L.rows) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (gc + e < L.cols) ptr[e] = (uint16_t)(v[i][e >> 1] >> (16 * (e & 1)));
                }
            }
        }
    };
    // two bf16 of a packed word as fp32, and back (round to nearest even)
    auto bf_lo = [](uint32_t w) { return __uint_as_float(w << 16); };
    auto bf_hi = [](uint32_t w) { return __uint_as_float(w & 0xffff0000u); };
    auto bf_pack = [](float lo, float hi) {
        const f32x2 v = {lo, hi};
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
    };
    auto store_rows = [&](const TileLoc& L, const u32x4 (&outv)[NI]) {
        if constexpr (OPT) {
            // W <- (1 - lr lambda) W - lr tau U, U the tile's bf16 result
            u32x4 wv[NI];
            load_rows(L, L.out, L.ld_out, L.vout, wv);
            const float step = args.lr * L.tau;
#pragma unroll
            for (int i = 0; i < NI; ++i)
#pragma unroll
                for (int x = 0; x < 4; ++x)
                    wv[i][x] = bf_pack(args.decay * bf_lo(wv[i][x]) - step * bf_lo(outv[i][x]),
                                       args.decay * bf_hi(wv[i][x]) - step * bf_hi(outv[i][x]));
            put_rows(L, L.out, L.ld_out, L.vout, wv);
        } else {
            put_rows(L, L.out, L.ld_out, L.vout, outv);
        }
    };
    // OPT, on the staged rows of the current tile: M <- beta M + G, stored
    // (bf16), and the lookahead from the stored M replaces G in `raw`
    auto step_prologue = [&](const TileLoc& L) {
        if constexpr (OPT) {
#pragma unroll
            for (int i = 0; i < NI; ++i)
#pragma unroll
                for (int x = 0; x < 4; ++x) {
                    const uint32_t g = raw[i][x];
                    const uint32_t m = bf_pack(args.beta * bf_lo(rawm[i][x]) + bf_lo(g),
                                               args.beta * bf_hi(rawm[i][x]) + bf_hi(g));
                    rawm[i][x] = m;
                    raw[i][x] = args.nesterov ? bf_pack(bf_lo(g) + args.beta * bf_lo(m), bf_hi(g) + args.beta * bf_hi(m))
                                              : m;
                }
            put_rows(L, L.mom, L.ld_in, L.vin, rawm);
        }
    };

    // Sum of squares of the tile from its packed bf16 words: per-lane fp32
    // dot products, then a fixed-order reduction over the lanes and the
    // waves of the tile (slot set `rs` of the exchange array).
    auto tile_sumsq = [&](const uint32_t (&W)[RB][NB][8], int rs) -> float {
        float v = 0.f;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    v = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, W[rb][q][i]),
                                                       __builtin_bit_cast(bf16x2, W[rb][q][i]), v, false);
        v = wave_sum_f32(v);
        if constexpr (SHARED) {
            if (lane == 0) s_red[rs][wave] = v;
            __syncthreads();
            v = s_red[rs][tslot * WT];
#pragma unroll
            for (int w = 1; w < WT; ++w) v += s_red[rs][tslot * WT + w];
        }
        return v;
    };

    int64_t local = (int64_t)blockIdx.x * TPW + tslot;
    if (local >= n_tiles) return;  // uniform over the waves that share a tile
    TileLoc cur;
    locate(local, cur);
    issue_loads(cur);
    // The previous tile's results wait in `outv` until this tile's rows have
    // left the prefetch registers: the prefetch wait then never waits on
    // stores (loads and stores share one memory counter).
    u32x4 outv[NI];
    TileLoc prv = cur;
    bool pending = false;
    int parity = 0;  // alternates the reduction slots between tiles

    for (;;) {
        const int64_t nlocal = local + (int64_t)gridDim.x * TPW;
        const bool has_next = nlocal < n_tiles;
        TileLoc nxt = cur;
        if (has_next) locate(nlocal, nxt);
        step_prologue(cur);

        // own rows into the row-major copy, then back as row pieces of packed
        // bf16 words; only this wave touches these rows until its first
        // step's barrier
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int row = 32 * p0 + RPI * i + io_row;
            if constexpr (PAIRS) {
                *reinterpret_cast<u32x2*>(rm + io_half(row, 0)) = u32x2{raw[i][0], raw[i][1]};
                *reinterpret_cast<u32x2*>(rm + io_half(row, 1)) = u32x2{raw[i][2], raw[i][3]};
            } else {
                *reinterpret_cast<u32x4*>(rm + io_lds(row)) = raw[i];
            }
        }
        if (pending) store_rows(prv, outv);
        if constexpr (EARLY) {
            if (has_next) issue_loads(nxt);  // in flight for the whole K loop
        }
        uint32_t W[RB][NB][8];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    if constexpr (PAIRS) {
                        if (g % 2 == 0) {
                            const u32x4 w = *reinterpret_cast<const u32x4*>(rm + 32 * (p0 + rb) * RS + 64 * q + rpB[g / 2]);
#pragma unroll
                            for (int x = 0; x < 4; ++x) W[rb][q][2 * g + x] = w[x];
                        }
                    } else {
                        const u32x2 w = *reinterpret_cast<const u32x2*>(rm + 32 * (p0 + rb) * RS + io_rp[g] + 64 * q);
                        W[rb][q][2 * g] = w[0];
                        W[rb][q][2 * g + 1] = w[1];
                    }
                }

        // Z_0 = |c|^(1/4) S / ||S||_F (Phi_K(0) = 0). The fp32 sum of squares
        // is exact enough whenever it lands in [2^-60, 2^100]; otherwise the
        // tile is first scaled by 2^-k, k the exponent of its largest entry
        // (exact, so Phi(2^e S) = Phi(S) bit for bit on either path), and the
        // same sum is taken again.
        float ss = tile_sumsq(W, 3 * parity);
        float sc = 0.f;
        if (ss != 0.f) {
            if (!(ss >= 0x1p-60f && ss <= 0x1p100f)) {
                uint32_t mb = 0;
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int q = 0; q < NB; ++q)
#pragma unroll
                        for (int i = 0; i < 8; ++i)
                            mb = max(mb, max(W[rb][q][i] & 0x7fffu, (W[rb][q][i] >> 16) & 0x7fffu));
                mb = wave_max_u32(mb);
                if constexpr (SHARED) {
                    if (lane == 0) s_red[3 * parity + 1][wave] = __uint_as_float(mb);
                    __syncthreads();
#pragma unroll
                    for (int w = 0; w < WT; ++w) mb = max(mb, __float_as_uint(s_red[3 * parity + 1][tslot * WT + w]));
                }
                const int k = (int)((mb >> 7) & 0xffu) - 127;
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int q = 0; q < NB; ++q)
#pragma unroll
                        for (int i = 0; i < 8; ++i) {
                            const float lo = ldexpf(__uint_as_float(W[rb][q][i] << 16), -k);
                            const float hi = ldexpf(__uint_as_float(W[rb][q][i] & 0xffff0000u), -k);
                            W[rb][q][i] = (__float_as_uint(hi) & 0xffff0000u) | (__float_as_uint(lo) >> 16);
                        }
                ss = tile_sumsq(W, 3 * parity + 2);
            }
            // ss = m 4^e with m in [1, 4): sc = |c|^(1/4) rsq(m) 2^-e. The
            // tile's scale reaches sc only through the exact factor 2^-e, which
            // keeps Phi(2^e S) = Phi(S) bit for bit; the hardware reciprocal
            // square root (about one ulp) is far inside the fp16 rounding of
            // the iterate.
            const uint32_t sb = __float_as_uint(ss);
            const int e = ((int)(sb >> 23) - 127) >> 1;
            const float m = __uint_as_float(sb - ((uint32_t)(2 * e) << 23));
            sc = ldexpf(args.zscale * __builtin_amdgcn_rsqf(m), -e);
        }
        parity ^= 1;
        f32x16 Z[RB][NB];
        // the result as packed bf16 row pieces (word 2g + i: columns 8g + 4lh + 2i, +1)
        uint32_t OB[RB][NB][8];
        auto pack_out = [&](const f32x16& z, uint32_t (&ob)[8]) {
#pragma unroll
            for (int i = 0; i < 8; ++i) ob[i] = pack2<Operand::BF16>(z[2 * i] * args.unscale, z[2 * i + 1] * args.unscale);
        };
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    Z[rb][q][2 * i] = __uint_as_float(W[rb][q][i] << 16) * sc;
                    Z[rb][q][2 * i + 1] = __uint_as_float(W[rb][q][i] & 0xffff0000u) * sc;
                }

        // The K steps of a 128-tile split over two waves, using the symmetry
        // of M and of aI + P (polynomials in H = Z Z^T): of the 16 blocks
        // of each, only the ten on and above the block diagonal are
        // computed, five per wave. Wave w owns row blocks r0 = 2w, r1 = r0+1
        // and computes blocks (r0,r0), (r0,r1), (r1,r1), (r0,o_w) and
        // (r1,o_{1-w}), o_0 < o_1 being the other wave's row blocks; the
        // other wave's cross blocks are then (o_0, r_{1-w}) and (o_1, r_w),
        // so each upper block is computed exactly once. Blocks are stored in
        // LDS as 32x32 fp16 arrays (64-byte rows, the Z copy's chunk
        // swizzle); a block needed in the other orientation is read with
        // ds_read_b64_tr_b16. The Gram blocks are those of M (the diagonal
        // ones carry the shift from the seed of their accumulators). Per step:
        //   Gram (r0,r0), part of (r0,r1), with the conversion of Z into
        //   operands | barrier | own Z rows to LDS + rest of the own Gram
        //   blocks | barrier | Gram cross blocks (+ own H conversions and
        //   stores) | cross H stores | P terms on own blocks | barrier | P
        //   terms on the other wave's blocks (+ conversions) | P stores | PZ
        //   over the own k-blocks | barrier | PZ over the other k-blocks.
        auto ns_steps_sym = [&]() {
          if constexpr (F16Shape<T, RB>::kSym) {
            static_assert(NB == 4 && RB == 2 && S == 2, "two waves of two 32-row blocks");
            const int w = p0 / RB, wo = 1 - w;
            const int ot = 2 * wo + w;      // o_t: the other block of this wave's (r0, .) cross block
            const int on = 2 * wo + 1 - w;  // o_{1-t}: that of (r1, .)
            // During the steps the Z copy and the blocks use a layout in which
            // an operand slot is one aligned 16-byte pair: within each 64-byte
            // segment, logical chunk c (columns 4c..4c+3) of row r sits at
            // pair ((c >> 2) * 2 + (c & 1)) ^ t(r), half (c >> 1) & 1, with
            // t(r) = ((r >> 1) ^ (r >> 2) ^ (r >> 4)) & 3. Slot s of lane
            // (li, lh) (chunks 4s + lh and 4s + 2 + lh) is then pair
            // (2s + lh) ^ t(li), so row pieces move with ds_read_b128 and
            // ds_write_b128; on gfx950 these, and the transposing reads of
            // the layout, are bank-conflict-free at row strides 320 and 64
            // bytes (measured with the LDS bank-conflict counter). The tile is
            // staged in the same layout (tsw, rpB and io_half above).
            auto phys = [&](int c, int r) { return 2 * ((((c >> 2) << 1) | (c & 1)) ^ tsw(r)) + ((c >> 1) & 1); };
            int bpB[S];
#pragma unroll
            for (int s = 0; s < S; ++s) bpB[s] = li * 64 + 16 * ((2 * s + lh) ^ tsw(li));
            int trB[S][2], btrB[S][2];
#pragma unroll
            for (int s = 0; s < S; ++s)
#pragma unroll
                for (int x = 0; x < 2; ++x) {
                    const int row = 16 * s + 8 * x + 4 * (grp16 >> 1) + ((lane & 15) >> 2);
                    const int chunk = 4 * (grp16 & 1) + (lane & 3);
                    trB[s][x] = row * RS + 8 * phys(chunk, row);
                    btrB[s][x] = row * 64 + 8 * phys(chunk, row);
                }
            uint8_t* const hb = reinterpret_cast<uint8_t*>(slots);
            // H blocks of wave v: 0 (r0,r0)', 1 (r0,r1), 2 (r1,r1)', 3 (r0,o_t),
            // 4 (r1,o_{1-t}), 5 (r1,r0); P blocks: 0 (r0,r1), 1 (r0,o_t), 2 (r1,o_{1-t})
            auto hblk = [&](int v, int e) -> uint8_t* { return hb + 2048 * (6 * v + e); };
            auto pblk = [&](int v, int e) -> uint8_t* { return hb + 2048 * (12 + 3 * v + e); };
            // slot s of a stored 32x32 block: its rows (lane = row), or the rows of its transpose
            auto blk_rows = [&](const uint8_t* b, int s) -> u32x4 { return *reinterpret_cast<const u32x4*>(b + bpB[s]); };
            auto blk_tr = [&](const uint8_t* b, int s) -> u32x4 {
                const u32x2 lo = tr_read(b + btrB[s][0]);
                const u32x2 hi = tr_read(b + btrB[s][1]);
                return u32x4{lo[0], lo[1], hi[0], hi[1]};
            };
            auto blk_put = [&](uint8_t* b, const u32x4 (&v)[S]) {
#pragma unroll
                for (int s = 0; s < S; ++s) *reinterpret_cast<u32x4*>(b + bpB[s]) = v[s];
            };
            // column pieces of Z's row block `br`, k half s, output block n; row pieces
            auto zcol = [&](int br, int s, int n) -> u32x4 {
                const uint8_t* const kb = rm + 32 * br * RS + 64 * n;
                const u32x2 lo = tr_read(kb + trB[s][0]);
                const u32x2 hi = tr_read(kb + trB[s][1]);
                return u32x4{lo[0], lo[1], hi[0], hi[1]};
            };
            auto zrow = [&](int br, int q, int s) -> u32x4 {
                return *reinterpret_cast<const u32x4*>(rm + 32 * br * RS + 64 * q + rpB[s]);
            };

            for (int k = 0; k < args.K; ++k) {
                // ---- Gram. The operands of the current Z are made here, each
                // right before its first product, and stored as this wave's rows
                // of the Z copy (no wave reads the copy after the previous
                // step's last barrier, see below).
                u32x4 Zop[RB][NB][S];
                f32x16 g[5];  // the diagonal blocks (r0, r0), (r1, r1) of M from the shift
#pragma unroll
                for (int e = 0; e < 5; ++e) g[e] = (e == 0 || e == 2) ? diag_m : f32x16{};
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int q = 0; q < NB; ++q)
#pragma unroll
                        for (int s = 0; s < S; ++s) {
                            Zop[rb][q][s] = make_slot<OP>(Z[rb][q], s);
                            if (rb == 0) g[0] = mma1<OP>(Zop[0][q][s], Zop[0][q][s], g[0]);
                            else g[1] = mma1<OP>(Zop[1][q][s], Zop[0][q][s], g[1]);
                            *reinterpret_cast<u32x4*>(rm + 32 * (p0 + rb) * RS + 64 * q + rpB[s]) = Zop[rb][q][s];
                            __builtin_amdgcn_sched_barrier(0);
                        }
#pragma unroll
                for (int q = 0; q < 2; ++q)
#pragma unroll
                    for (int s = 0; s < S; ++s) g[2] = mma1<OP>(Zop[1][q][s], Zop[1][q][s], g[2]);
                __syncthreads();

                // ---- Gram cross blocks (r0, o_t), (r1, o_{1-t}) from the other
                // wave's Z rows, read PD iterations ahead (the last own products
                // cover the first reads); the own blocks' conversions and
                // stores ride along
                constexpr int PD = 3;
                u32x4 rq[PD][2];
#pragma unroll
                for (int d = 0; d < PD; ++d) {
                    rq[d][0] = zrow(ot, d / S, d % S);
                    rq[d][1] = zrow(on, d / S, d % S);
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int q = 2; q < NB; ++q)
#pragma unroll
                    for (int s = 0; s < S; ++s) g[2] = mma1<OP>(Zop[1][q][s], Zop[1][q][s], g[2]);
                __builtin_amdgcn_sched_barrier(0);
                u32x4 hs[5][S], la1[S];  // hs[0], hs[2]: diagonal blocks of M; la1: H[r1, r0]
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    const int q = it / S, s = it % S;
                    const u32x4 c0 = rq[it % PD][0], c1 = rq[it % PD][1];
                    if (it + PD < IT) {
                        rq[it % PD][0] = zrow(ot, (it + PD) / S, (it + PD) % S);
                        rq[it % PD][1] = zrow(on, (it + PD) / S, (it + PD) % S);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                    g[3] = mma1<OP>(c0, Zop[0][q][s], g[3]);
                    g[4] = mma1<OP>(c1, Zop[1][q][s], g[4]);
                    if constexpr (CMODE != 2) {
                        if (it == 0) {
#pragma unroll
                            for (int x = 0; x < S; ++x) hs[0][x] = make_slot<OP>(g[0], x);
                        } else if (it == 1) {
                            blk_put(hblk(w, 0), hs[0]);
                        } else if (it == 2) {
#pragma unroll
                            for (int x = 0; x < S; ++x) hs[1][x] = make_slot<OP>(g[1], x);
                        } else if (it == 3) {
                            blk_put(hblk(w, 1), hs[1]);
#pragma unroll
                            for (int x = 0; x < S; ++x) hs[2][x] = make_slot<OP>(g[2], x);
                        } else if (it == 4) {
                            blk_put(hblk(w, 2), hs[2]);
                        } else if (it == 5) {
#pragma unroll
                            for (int x = 0; x < S; ++x) la1[x] = blk_tr(hblk(w, 1), x);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }

                u32x4 pop[5][S];
                f32x16 pa[5];
                auto pconv = [&](int e) {
#pragma unroll
                    for (int x = 0; x < S; ++x) {
                        if constexpr (CMODE == 0) pop[e][x] = make_slot<OP>(pa[e], x);
                        else pop[e][x] = make_slot<OP>(-pa[e], x);
                    }
                };
                if constexpr (CMODE != 2) {
                    // ---- P (as acc = M M + sigma a' I): block (i, j) accumulates
                    // M[j, k] x M[i, k] over the k-blocks (M and H share their
                    // off-diagonal blocks). Terms on this wave's blocks first;
                    // the cross blocks' conversions and stores ride along.
                    pa[0] = diag_a;
                    pa[1] = f32x16{};
                    pa[2] = diag_a;
                    pa[3] = f32x16{};
                    pa[4] = f32x16{};
                    u32x4 lb1[S], lb6[S];  // H[o_t, r0], H[o_{1-t}, r1]
#pragma unroll
                    for (int s = 0; s < S; ++s) {
                        pa[0] = mma1<OP>(hs[0][s], hs[0][s], pa[0]);  // k = r0
                        pa[1] = mma1<OP>(hs[2][s], hs[1][s], pa[1]);  // k = r1
                        pa[2] = mma1<OP>(hs[2][s], hs[2][s], pa[2]);  // k = r1
                        pa[0] = mma1<OP>(hs[1][s], hs[1][s], pa[0]);  // k = r1
                        pa[1] = mma1<OP>(la1[s], hs[0][s], pa[1]);    // k = r0
                        pa[2] = mma1<OP>(la1[s], la1[s], pa[2]);      // k = r0
                        if (s == 0) {
                            blk_put(hblk(w, 5), la1);
#pragma unroll
                            for (int x = 0; x < S; ++x) hs[3][x] = make_slot<OP>(g[3], x);
                            blk_put(hblk(w, 3), hs[3]);
                        } else {
#pragma unroll
                            for (int x = 0; x < S; ++x) hs[4][x] = make_slot<OP>(g[4], x);
                            blk_put(hblk(w, 4), hs[4]);
#pragma unroll
                            for (int x = 0; x < S; ++x) {
                                lb1[x] = blk_tr(hblk(w, 3), x);
                                lb6[x] = blk_tr(hblk(w, 4), x);
                            }
                        }
                        __builtin_amdgcn_sched_barrier(0);
                    }
#pragma unroll
                    for (int s = 0; s < S; ++s) {
                        pa[0] = mma1<OP>(hs[3][s], hs[3][s], pa[0]);  // k = o_t
                        pa[2] = mma1<OP>(hs[4][s], hs[4][s], pa[2]);  // k = o_{1-t}
                    }
                    __builtin_amdgcn_sched_barrier(0);
                    __syncthreads();
                    // the other wave's blocks; two own terms cover their reads
                    u32x4 la2[S], la3[S], lb2[S], lb3[S], lb4[S], lb5[S], lb7[S], lb8[S];
#pragma unroll
                    for (int s = 0; s < S; ++s) {
                        la2[s] = blk_tr(hblk(wo, 4 - w), s);     // H[r0, o_{1-t}]
                        la3[s] = blk_tr(hblk(wo, 3 + w), s);     // H[r1, o_t]
                    }
#pragma unroll
                    for (int s = 0; s < S; ++s) {
                        lb2[s] = blk_rows(hblk(wo, 3 + w), s);      // H[o_t, r1]
                        lb3[s] = blk_rows(hblk(wo, 2 * w), s);      // M[o_t, o_t]
                        lb4[s] = blk_rows(hblk(wo, w ? 5 : 1), s);  // H[o_t, o_{1-t}]
                        lb7[s] = blk_rows(hblk(wo, w ? 1 : 5), s);  // H[o_{1-t}, o_t]
                        lb5[s] = blk_rows(hblk(wo, 4 - w), s);      // H[o_{1-t}, r0]
                        lb8[s] = blk_rows(hblk(wo, 2 - 2 * w), s);  // M[o_{1-t}, o_{1-t}]
                    }
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int s = 0; s < S; ++s) {
                        pa[3] = mma1<OP>(lb1[s], hs[0][s], pa[3]);    // (r0, o_t), k = r0
                        pa[4] = mma1<OP>(lb6[s], hs[2][s], pa[4]);    // (r1, o_{1-t}), k = r1
                    }
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int s = 0; s < S; ++s) {
                        pa[0] = mma1<OP>(la2[s], la2[s], pa[0]);    // k = o_{1-t}
                        pa[1] = mma1<OP>(la3[s], hs[3][s], pa[1]);  // k = o_t
                        pa[2] = mma1<OP>(la3[s], la3[s], pa[2]);    // k = o_t
                        pa[1] = mma1<OP>(hs[4][s], la2[s], pa[1]);  // k = o_{1-t}
                        __builtin_amdgcn_sched_barrier(0);
                    }
#pragma unroll
                    for (int s = 0; s < S; ++s) {
                        pa[3] = mma1<OP>(lb2[s], hs[1][s], pa[3]);  // (r0, o_t), k = r1
                        pa[4] = mma1<OP>(lb5[s], la1[s], pa[4]);    // (r1, o_{1-t}), k = r0
                        pa[3] = mma1<OP>(lb3[s], hs[3][s], pa[3]);  // k = o_t
                        pa[4] = mma1<OP>(lb7[s], la3[s], pa[4]);    // k = o_t
                        pa[3] = mma1<OP>(lb4[s], la2[s], pa[3]);    // k = o_{1-t}
                        pa[4] = mma1<OP>(lb8[s], hs[4][s], pa[4]);  // k = o_{1-t}
                        if (s == 0) {
                            pconv(0);
                            pconv(1);
                        } else {
                            pconv(2);
                            blk_put(pblk(w, 0), pop[1]);
                        }
                        __builtin_amdgcn_sched_barrier(0);
                    }
                } else {
                    // c = 0: aI + P = a I + b H, straight from the Gram blocks
#pragma unroll
                    for (int e = 0; e < 5; ++e) pa[e] = (e == 0 || e == 2) ? g[e] * args.bq + diag_a : g[e] * args.bq;
#pragma unroll
                    for (int e = 0; e < 3; ++e)
#pragma unroll
                        for (int x = 0; x < S; ++x) pop[e][x] = make_slot<OP>(pa[e], x);
                    blk_put(pblk(w, 0), pop[1]);
                }

                // ---- Z <- (a I + P) Z over the k-blocks r0, r1, o_t, o_{1-t}
                // (two k halves each). Before the barrier: every product on this
                // wave's blocks of aI + P ((aI + P)[r1, r0] is the transpose of its
                // own (r0, r1) block) but one k half, with the cross blocks'
                // conversions and stores riding along; the column pieces of the
                // other wave's rows stay in registers for the two products on
                // the other wave's blocks after it. So no wave reads the Z copy
                // after the barrier, and the next step stores its rows at once.
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int n = 0; n < NB; ++n) Z[rb][n] = f32x16{};
                u32x4 lp[3][S];  // (aI + P)[r1, r0], [r0, o_{1-t}], [r1, o_t]
#pragma unroll
                for (int s = 0; s < S; ++s) lp[0][s] = blk_tr(pblk(w, 0), s);
                // (k-block, half) read order; pieces of o_t and o_{1-t} are kept
                constexpr int NPZ = 8;
                auto pz_blk = [&](int it) -> int { return it < 2 ? p0 : (it == 2 ? p0 + 1 : (it < 5 ? ot : (it < 7 ? on : p0 + 1))); };
                auto pz_half = [&](int it) -> int { return it < 2 ? it : (it == 2 ? 0 : (it < 5 ? it - 3 : (it < 7 ? it - 5 : 1))); };
                u32x4 kept[2][S][NB];  // column pieces of o_t, o_{1-t}
                u32x4 nxt[NB];
#pragma unroll
                for (int n = 0; n < NB; ++n) nxt[n] = zcol(pz_blk(0), pz_half(0), n);
#pragma unroll
                for (int it = 0; it < NPZ; ++it) {
                    const int s = pz_half(it);
                    if (it == 7) {
                        __syncthreads();
#pragma unroll
                        for (int x = 0; x < S; ++x) {
                            lp[1][x] = blk_tr(pblk(wo, 2 - w), x);
                            lp[2][x] = blk_tr(pblk(wo, 1 + w), x);
                        }
                    }
                    u32x4 cur[NB];
#pragma unroll
                    for (int n = 0; n < NB; ++n) cur[n] = nxt[n];
                    if (it + 1 < NPZ) {
#pragma unroll
                        for (int n = 0; n < NB; ++n) nxt[n] = zcol(pz_blk(it + 1), pz_half(it + 1), n);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                    if (it < 3 || it == 7) {  // own k-blocks, both rows
                        const u32x4 a0 = it < 2 ? pop[0][s] : pop[1][s];
                        const u32x4 a1 = it < 2 ? lp[0][s] : pop[2][s];
#pragma unroll
                        for (int n = 0; n < NB; ++n) {
                            Z[0][n] = mma1<OP>(cur[n], a0, Z[0][n]);
                            Z[1][n] = mma1<OP>(cur[n], a1, Z[1][n]);
                        }
                    } else if (it < 5) {  // o_t: row r0 on this wave's (r0, o_t) block
#pragma unroll
                        for (int n = 0; n < NB; ++n) {
                            kept[0][s][n] = cur[n];
                            Z[0][n] = mma1<OP>(cur[n], pop[3][s], Z[0][n]);
                        }
                    } else {  // o_{1-t}: row r1 on this wave's (r1, o_{1-t}) block
#pragma unroll
                        for (int n = 0; n < NB; ++n) {
                            kept[1][s][n] = cur[n];
                            Z[1][n] = mma1<OP>(cur[n], pop[4][s], Z[1][n]);
                        }
                    }
                    if (it == 0) {
                        if constexpr (CMODE != 2) pconv(3);
                        else {
#pragma unroll
                            for (int x = 0; x < S; ++x) pop[3][x] = make_slot<OP>(pa[3], x);
                        }
                    } else if (it == 1) {
                        if constexpr (CMODE != 2) pconv(4);
                        else {
#pragma unroll
                            for (int x = 0; x < S; ++x) pop[4][x] = make_slot<OP>(pa[4], x);
                        }
                        blk_put(pblk(w, 1), pop[3]);
                    } else if (it == 2) {
                        blk_put(pblk(w, 2), pop[4]);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
                // the other wave's blocks: (aI + P)[r1, o_t] and [r0, o_{1-t}]
#pragma unroll
                for (int s = 0; s < S; ++s) {
#pragma unroll
                    for (int n = 0; n < NB; ++n) {
                        Z[1][n] = mma1<OP>(kept[0][s][n], lp[2][s], Z[1][n]);
                        Z[0][n] = mma1<OP>(kept[1][s][n], lp[1][s], Z[0][n]);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            // the other wave's last reads of this wave's rows come before the
            // write-back reuses them
            if (args.K > 0) __syncthreads();
          }
        };

        // The K steps of a 256-tile (one tile per CU, four waves of two row
        // blocks each). Its fp16 copy fills the LDS, so H is never exchanged:
        // each step is evaluated in the equivalent chain form
        //     Y = sigma M Z,   Z <- a' Z + M Y,
        // with M's own rows kept in registers. Column block N of Y depends
        // only on column block N of Z, so Y replaces Z in the row-major copy
        // one column half at a time:
        //   Z own rows to LDS | barrier | Gram | Y, first half | barrier |
        //   Y first half to LDS | Y, second half | barrier | Y second half to
        //   LDS | MY, first half | barrier | MY, second half.
        // Products run on groups of NG column blocks, which bounds the
        // accumulators to 64 registers; each MY group is converted at once
        // into the next step's fp16 operands, from which the bf16 output is
        // rounded after the last step (for K = 0 too, so that no fp32 copy of
        // the tile stays live across the steps). The barrier at the top of each later step keeps
        // the other waves' reads of Y ahead of this wave's overwrite of its rows.
        auto ns_steps_chain = [&]() {
          if constexpr (F16Shape<T, RB>::kChain) {
            constexpr int NG = 2;       // column blocks per product group
            constexpr int NGR = NB / NG;
            constexpr int NH = NB / 2;  // column blocks per half
            u32x4 Zop[RB][NB][S];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int q = 0; q < NB; ++q)
#pragma unroll
                    for (int s = 0; s < S; ++s) Zop[rb][q][s] = make_slot<OP>(Z[rb][q], s);
            // own rows (row pieces) of a 16-bit operand matrix into the copy
            auto put_rows = [&](const u32x4 (&V)[RB][NB][S], int n0, int n1) {
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int N = n0; N < n1; ++N)
#pragma unroll
                        for (int g = 0; g < 4; ++g)
                            *reinterpret_cast<u32x2*>(rm + 32 * (p0 + rb) * RS + rp_off[g] + 64 * N) =
                                u32x2{V[rb][N][g >> 1][(g & 1) * 2], V[rb][N][g >> 1][(g & 1) * 2 + 1]};
            };
            auto col_piece = [&](int it, int N) -> u32x4 {
                const int jk = it / S, s = it % S;
                const uint8_t* const kb = rm + 32 * ((p0 + jk) % NB) * RS + 64 * N;
                const u32x2 lo = tr_read(kb + tr_off[s][0]);
                const u32x2 hi = tr_read(kb + tr_off[s][1]);
                return u32x4{lo[0], lo[1], hi[0], hi[1]};
            };
            // acc[rb][n] += sum over the rotated k-blocks of col(., n0 + n) x B(rb, jk, s)
            auto col_product = [&](f32x16 (&acc)[RB][NG], int n0, auto&& bop) {
                u32x4 nxt_op[NG];
#pragma unroll
                for (int n = 0; n < NG; ++n) nxt_op[n] = col_piece(0, n0 + n);
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    const int jk = it / S, s = it % S;
                    u32x4 cur_op[NG];
#pragma unroll
                    for (int n = 0; n < NG; ++n) cur_op[n] = nxt_op[n];
                    if (it + 1 < IT) {
#pragma unroll
                        for (int n = 0; n < NG; ++n) nxt_op[n] = col_piece(it + 1, n0 + n);
                    }
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int n = 0; n < NG; ++n)
#pragma unroll
                        for (int rb = 0; rb < RB; ++rb) acc[rb][n] = mma1<OP>(cur_op[n], bop(rb, jk, s), acc[rb][n]);
                    __builtin_amdgcn_sched_barrier(0);
                }
            };
            for (int k = 0; k < args.K; ++k) {
                if (k > 0) __syncthreads();
                put_rows(Zop, 0, NB);
                __syncthreads();

                // ---- M = Z Z^T + (sigma b' / 2) I by groups of NG rotated column
                // blocks (b H for c = 0); G[rb][jj] is block (p0 + rb, (p0 + NG gq
                // + jj) mod NB), diagonal for NG gq + jj = rb
                u32x4 Hop[RB][NB][S];
#pragma unroll
                for (int gq = 0; gq < NGR; ++gq) {
                    f32x16 G[RB][NG];
#pragma unroll
                    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                        for (int jj = 0; jj < NG; ++jj) G[rb][jj] = NG * gq + jj == rb ? diag_m : f32x16{};
                    auto opa = [&](int j, int q, int s) -> u32x4 {
                        return j < RB ? Zop[j < RB ? j : 0][q][s] : rowpiece(rm_row[j < RB ? 0 : j - RB], q, s);
                    };
                    u32x4 nxt_op[NG];
#pragma unroll
                    for (int jj = 0; jj < NG; ++jj) nxt_op[jj] = opa(NG * gq + jj, 0, 0);
#pragma unroll
                    for (int it = 0; it < IT; ++it) {
                        const int q = it / S, s = it % S;
                        u32x4 cur_op[NG];
#pragma unroll
                        for (int jj = 0; jj < NG; ++jj) cur_op[jj] = nxt_op[jj];
                        if (it + 1 < IT) {
#pragma unroll
                            for (int jj = 0; jj < NG; ++jj) nxt_op[jj] = opa(NG * gq + jj, (it + 1) / S, (it + 1) % S);
                        }
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int jj = 0; jj < NG; ++jj)
#pragma unroll
                            for (int rb = 0; rb < RB; ++rb) G[rb][jj] = mma1<OP>(cur_op[jj], Zop[rb][q][s], G[rb][jj]);
                        __builtin_amdgcn_sched_barrier(0);
                    }
#pragma unroll
                    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                        for (int jj = 0; jj < NG; ++jj) {
                            const int j = NG * gq + jj;
                            const f32x16 gj = CMODE == 2 ? G[rb][jj] * args.bq : G[rb][jj];
#pragma unroll
                            for (int s = 0; s < S; ++s) Hop[rb][j][s] = make_slot<OP>(gj, s);
                        }
                }
                auto hb = [&](int rb, int jk, int s) -> u32x4 { return Hop[rb][jk][s]; };
                // a' Z (a Z for c = 0; fp16 state, exact products) as the seed of
                // the last product
                auto seed = [&](f32x16 (&acc)[RB][NG], int n0) {
                    const float sa = CMODE == 2 ? args.a : args.am;
#pragma unroll
                    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                        for (int n = 0; n < NG; ++n)
#pragma unroll
                            for (int s = 0; s < S; ++s)
#pragma unroll
                                for (int w = 0; w < 4; ++w) {
                                    // (copied out first: a bit cast of a vector element
                                    // would read the vector's first element)
                                    // (fma with a zero addend: one mixed-precision
                                    // instruction per value, the same rounding)
                                    const uint32_t wv = Zop[rb][n0 + n][s][w];
                                    const f16x2 pr = __builtin_bit_cast(f16x2, wv);
                                    acc[rb][n][8 * s + 2 * w] = __builtin_fmaf(sa, (float)pr[0], 0.f);
                                    acc[rb][n][8 * s + 2 * w + 1] = __builtin_fmaf(sa, (float)pr[1], 0.f);
                                }
                };
                // a finished group of Z becomes next step's operands (after the
                // last step, the output is rounded from these fp16 values)
                auto finish = [&](f32x16 (&acc)[RB][NG], int n0) {
#pragma unroll
                    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                        for (int n = 0; n < NG; ++n)
#pragma unroll
                            for (int s = 0; s < S; ++s) Zop[rb][n0 + n][s] = make_slot<OP>(acc[rb][n], s);
                };
                auto hy_group = [&](int gq) {
                    f32x16 acc[RB][NG];
                    seed(acc, NG * gq);
                    col_product(acc, NG * gq, hb);
                    finish(acc, NG * gq);
                };
                if constexpr (CMODE == 2) {
                    // c = 0: Z <- a Z + b H Z, the H Z product reading Z itself
#pragma unroll
                    for (int gq = 0; gq < NGR; ++gq) hy_group(gq);
                } else {
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        u32x4 Yop[RB][NB][S];  // (only column half h is set)
#pragma unroll
                        for (int gq = h * NGR / 2; gq < (h + 1) * NGR / 2; ++gq) {
                            f32x16 acc[RB][NG];
#pragma unroll
                            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                                for (int n = 0; n < NG; ++n) acc[rb][n] = f32x16{};
                            col_product(acc, NG * gq, hb);
#pragma unroll
                            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                                for (int n = 0; n < NG; ++n)
#pragma unroll
                                    for (int s = 0; s < S; ++s)
                                        Yop[rb][NG * gq + n][s] = make_slot<OP>(CMODE == 1 ? -acc[rb][n] : acc[rb][n], s);
                        }
                        __syncthreads();  // every wave is done reading this column half of Z
                        put_rows(Yop, NH * h, NH * (h + 1));
                    }
                    // Z <- a' Z + M Y, by column halves
#pragma unroll
                    for (int gq = 0; gq < NGR / 2; ++gq) hy_group(gq);
                    __syncthreads();  // the second half of Y is visible
#pragma unroll
                    for (int gq = NGR / 2; gq < NGR; ++gq) hy_group(gq);
                }
            }
            // the other waves' last reads of this wave's rows come before the
            // write-back reuses them
            {
                if (args.K > 0) __syncthreads();
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int q = 0; q < NB; ++q)
#pragma unroll
                        for (int s = 0; s < S; ++s)
#pragma unroll
                            for (int w = 0; w < 4; ++w) {
                                const uint32_t wv = Zop[rb][q][s][w];
                                const f16x2 pr = __builtin_bit_cast(f16x2, wv);
                                OB[rb][q][4 * s + w] = pack2<Operand::BF16>(__builtin_fmaf((float)pr[0], args.unscale, 0.f),
                                                                            __builtin_fmaf((float)pr[1], args.unscale, 0.f));
                            }
            }
          }
        };

        // One Newton-Schulz step.
        auto ns_step = [&]() {
            // SYM64: 32x32 fp16 blocks in LDS in the pair layout of the
            // symmetric 128-tile step (64-byte rows); a block stored from its
            // row pieces is read back transposed with ds_read_b64_tr_b16
            uint8_t* const sblk = reinterpret_cast<uint8_t*>(s_slots) + (SYM64 ? tslot * 4096 : 0);
            auto sym_put = [&](uint8_t* b, const u32x4 (&v)[S]) {
#pragma unroll
                for (int x = 0; x < S; ++x)
                    *reinterpret_cast<u32x4*>(b + li * 64 + 16 * ((2 * x + lh) ^ tsw(li))) = v[x];
            };
            auto sym_tr = [&](const uint8_t* b, int x) -> u32x4 {
                auto phys = [&](int c, int r) { return 2 * ((((c >> 2) << 1) | (c & 1)) ^ tsw(r)) + ((c >> 1) & 1); };
                u32x2 h[2];
#pragma unroll
                for (int y = 0; y < 2; ++y) {
                    const int row = 16 * x + 8 * y + 4 * (grp16 >> 1) + ((lane & 15) >> 2);
                    const int chunk = 4 * (grp16 & 1) + (lane & 3);
                    h[y] = tr_read(b + row * 64 + 8 * phys(chunk, row));
                }
                return u32x4{h[0][0], h[0][1], h[1][0], h[1][1]};
            };
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

            // M = Z Z^T + (sigma b' / 2) I (H itself for c = 0): G[rb][j] is the
            // row piece of block (p0 + rb, (p0 + j) mod NB), diagonal for j = rb.
            // Iteration it = (q, s) reads the other waves' row pieces (q, s) from
            // the row-major copy; those of iteration it + 1 are requested before
            // its MFMAs issue.
            f32x16 G[RB][NB];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int j = 0; j < NB; ++j) G[rb][j] = j == rb ? diag_m : f32x16{};
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
                        for (int rb = 0; rb < RB; ++rb) {
                            if (SYM64 && rb == 1 && j == 0) continue;  // the transpose of block (0, 1)
                            G[rb][j] = mma1<OP>(opa, Zop[rb][q][s], G[rb][j]);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }

            u32x4 Pop[RB][NB][S];  // own rows of P (rotated k-blocks), fp16
            if constexpr (CMODE != 2) {
                u32x4 Hop[RB][NB][S];
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int j = 0; j < NB; ++j)
#pragma unroll
                        for (int s = 0; s < S; ++s)
                            if (!(SYM64 && rb == 1 && j == 0)) Hop[rb][j][s] = make_slot<OP>(G[rb][j], s);
                if constexpr (SYM64) {
                    // M(1, 0) = M(0, 1)^T
                    sym_put(sblk, Hop[0][1]);
#pragma unroll
                    for (int s = 0; s < S; ++s) Hop[1][0][s] = sym_tr(sblk, s);
                }
                if constexpr (SHARED) {
                    // the M slots were last read before the previous step's final barrier
#pragma unroll
                    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                        for (int j = 0; j < NB; ++j)
#pragma unroll
                            for (int s = 0; s < S; ++s)
                                slots[(((p0 + rb) * NB + (p0 + j) % NB) * S + s) * 64 + lane] = Hop[rb][j][s];
                    __syncthreads();
                }
                // acc = M M + sigma a' I, so that sigma acc = a I + P: acc[rb][j]
                // is block (p0 + rb, (p0 + j) mod NB), the diagonal blocks (j = rb)
                // start from sigma a' I; iteration it = (jk, s) runs over the
                // rotated k-blocks (p0 + jk) mod NB.
                f32x16 acc[RB][NB];
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int j = 0; j < NB; ++j) acc[rb][j] = j == rb ? diag_a : f32x16{};
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
                            if (SYM64 && rb == 1 && j == 0) continue;  // aI + P is symmetric too
                            acc[rb][j] = mma1<OP>(opa, Hop[rb][jk][s], acc[rb][j]);
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
                            if (SYM64 && rb == 1 && j == 0) continue;
                            if constexpr (CMODE == 0) Pop[rb][j][s] = make_slot<OP>(acc[rb][j], s);
                            else Pop[rb][j][s] = make_slot<OP>(-acc[rb][j], s);
                        }
                if constexpr (SYM64) {
                    // (aI + P)(1, 0) = (aI + P)(0, 1)^T
                    sym_put(sblk + 2048, Pop[0][1]);
#pragma unroll
                    for (int s = 0; s < S; ++s) Pop[1][0][s] = sym_tr(sblk + 2048, s);
                }
            } else {
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int j = 0; j < NB; ++j) {
                        const f32x16 pj = j == rb ? G[rb][j] * args.bq + diag_a : G[rb][j] * args.bq;
#pragma unroll
                        for (int s = 0; s < S; ++s) Pop[rb][j][s] = make_slot<OP>(pj, s);
                    }
            }


            // Z <- (a I + P) Z, from zero accumulators; iteration it = (jk, s)
            // needs the column pieces of k-block (p0 + jk) mod NB for every
            // output block N (two transposing reads each), shared by the RB
            // owned row blocks.
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int N = 0; N < NB; ++N) Z[rb][N] = f32x16{};
            {
                auto col_piece = [&](int it, int N) -> u32x4 {
                    const int jk = it / S, s = it % S;
                    const uint8_t* const kb = rm + 32 * ((p0 + jk) % NB) * RS + 64 * N;
                    const u32x2 lo = tr_read(kb + tr_off[s][0]);
                    const u32x2 hi = tr_read(kb + tr_off[s][1]);
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
        if constexpr (F16Shape<T, RB>::kSym) ns_steps_sym();
        else if constexpr (F16Shape<T, RB>::kChain) ns_steps_chain();
        else
            for (int k = 0; k < args.K; ++k) ns_step();

        // row pieces (scaled back, rounded to bf16) into the own rows of the
        // row-major copy, then read back as whole 16-byte row chunks
        if constexpr (!F16Shape<T, RB>::kChain) {  // (the chain step packs its own output)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int q = 0; q < NB; ++q) pack_out(Z[rb][q], OB[rb][q]);
        }
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    if constexpr (PAIRS) {
                        if (g % 2 == 0)
                            *reinterpret_cast<u32x4*>(rm + 32 * (p0 + rb) * RS + 64 * q + rpB[g / 2]) =
                                u32x4{OB[rb][q][2 * g], OB[rb][q][2 * g + 1], OB[rb][q][2 * g + 2], OB[rb][q][2 * g + 3]};
                    } else {
                        *reinterpret_cast<u32x2*>(rm + 32 * (p0 + rb) * RS + io_rp[g] + 64 * q) =
                            u32x2{OB[rb][q][2 * g], OB[rb][q][2 * g + 1]};
                    }
                }
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int row = 32 * p0 + RPI * i + io_row;
            if constexpr (PAIRS) {
                const u32x2 lo = *reinterpret_cast<const u32x2*>(rm + io_half(row, 0));
                const u32x2 hi = *reinterpret_cast<const u32x2*>(rm + io_half(row, 1));
                outv[i] = u32x4{lo[0], lo[1], hi[0], hi[1]};
            } else {
                outv[i] = *reinterpret_cast<const u32x4*>(rm + io_lds(row));
            }
        }
        prv = cur;
        pending = true;
        // (raw is defined on both paths, so the values staged at the top of
        // this round are dead across its steps; the hint keeps the zeroing,
        // once per wave, off the path of every other round)
        if constexpr (!EARLY) {
            if (__builtin_expect(has_next, 1)) {
                issue_loads(nxt);
            } else {
#pragma unroll
                for (int i = 0; i < NI; ++i) raw[i] = u32x4{};
            }
        }
        if (!has_next) break;
        cur = nxt;
        local = nlocal;
    }
    store_rows(prv, outv);
    };
    if constexpr (F16Shape<T, RB>::kSym) {
        if (p0_rt == 0) tile_loop(std::integral_constant<int, 0>{});
        else tile_loop(std::integral_constant<int, 1>{});
    } else {
        tile_loop(std::integral_constant<int, -1>{});
    }
}

constexpr int kMaxDevices = 64;

template <int T, int RB, int CMODE, bool OPT = false>
hipError_t launch_f16(const KernelArgs& args, hipStream_t stream)
{
    constexpr int TPW = F16Shape<T, RB>::TPW;
    constexpr int NT = F16Shape<T, RB>::kThreads;
    static std::atomic<int> resident[kMaxDevices];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    int cap = resident[dev].load(std::memory_order_relaxed);
    if (cap == 0) {
        int per_cu = 0, cus = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, ns_tiled_f16_kernel<T, RB, CMODE, OPT>, NT, 0);
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
    hipLaunchKernelGGL((ns_tiled_f16_kernel<T, RB, CMODE, OPT>), dim3(grid), dim3(NT), 0, stream, args);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_ns_tiled_f16(int T, const KernelArgs& args, hipStream_t stream)
{
    if (args.step) {  // the optimizer step (c > 0, T <= 128; has_step_kernel)
        if (!(args.c > 0.f)) return hipErrorInvalidValue;
        switch (T) {
        case 32: return launch_f16<32, 1, 0, true>(args, stream);
        case 64: return launch_f16<64, 2, 0, true>(args, stream);
        case 128: return launch_f16<128, 2, 0, true>(args, stream);
        default: return hipErrorInvalidValue;
        }
    }
    const int cm = args.c > 0.f ? 0 : (args.c < 0.f ? 1 : 2);
    switch (T * 4 + cm) {
    case 32 * 4 + 0: return launch_f16<32, 1, 0>(args, stream);
    case 32 * 4 + 1: return launch_f16<32, 1, 1>(args, stream);
    case 32 * 4 + 2: return launch_f16<32, 1, 2>(args, stream);
    case 64 * 4 + 0: return launch_f16<64, 2, 0>(args, stream);
    case 64 * 4 + 1: return launch_f16<64, 2, 1>(args, stream);
    case 64 * 4 + 2: return launch_f16<64, 2, 2>(args, stream);
    case 128 * 4 + 0: return launch_f16<128, 2, 0>(args, stream);
    case 128 * 4 + 1: return launch_f16<128, 2, 1>(args, stream);
    case 128 * 4 + 2: return launch_f16<128, 2, 2>(args, stream);
    case 256 * 4 + 0: return launch_f16<256, 2, 0>(args, stream);
    case 256 * 4 + 1: return launch_f16<256, 2, 1>(args, stream);
    case 256 * 4 + 2: return launch_f16<256, 2, 2>(args, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace himuon
