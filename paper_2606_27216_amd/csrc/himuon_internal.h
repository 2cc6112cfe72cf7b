// Internal contract between the host planner (himuon_api.cpp) and the
// gfx950 kernel family (ns_tiled_kernels.hip). Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

namespace himuon {

// One entry per matrix in a call; the table lives in the caller's workspace.
// Global tile ids are dense: matrix m owns [tile_begin, tile_begin + R*C),
// numbered row-major over its R x C tile grid.
struct alignas(64) MatDesc {
    const void* in;
    void* out;
    int64_t rows, cols;
    int64_t ld_in, ld_out;
    int64_t tile_begin;
    int32_t tiles_c;  // C = ceil(cols / T)
    int32_t flags;    // MAT_VEC_IN / MAT_VEC_OUT
};
static_assert(sizeof(MatDesc) == 64, "descriptor layout");

// Base pointer and leading dimension allow 16-byte accesses at every column
// that is a multiple of 8 (bf16) or 4 (f32).
constexpr int32_t MAT_VEC_IN = 1;
constexpr int32_t MAT_VEC_OUT = 2;

enum class Storage : int { F32 = 0, BF16 = 1 };
enum class Operand : int { F32 = 1, F16 = 2, BF16 = 3 };

// The optimizer step of Alg. 1 fused into the fp16 tile kernels, per
// matrix: `in` is the gradient G, `out` the weights W (updated in place),
// `mom` the momentum M (layout of `in`, updated in place), tau the update
// scale of eq. (scaled_update).
struct alignas(16) OptDesc {
    void* mom;
    float tau;
    int32_t pad_;
};
static_assert(sizeof(OptDesc) == 16, "optimizer descriptor layout");

// Descriptors a launch carries in its own arguments: a call of at most this
// many matrices copies no table to the device before its kernels (2.5 KiB of
// kernel arguments).
constexpr int kInlineMats = 32;

// Kernel arguments of one chunk launch: tiles [tile_begin, tile_end).
struct KernelArgs {
    // The descriptor tables in device memory, or null: then they are
    // inline_descs / inline_odescs below.
    const MatDesc* descs;
    const OptDesc* odescs;
    // 1: the launch is an optimizer step (OptDesc per matrix). The tile
    // staging forms M <- beta M + G (stored, rounded to bf16) and the
    // lookahead G + beta M (nesterov) or M as the tile's input; the
    // write-back stores W <- decay W - lr tau U.
    int32_t step;
    float beta, decay, lr;
    int32_t nesterov;
    int64_t tile_begin;
    int64_t tile_end;
    int32_t n_mats;
    int32_t K;
    float a, b, c;
    float b_over_c;  // b / c, used when c != 0
    // Rescaled state Z = X |c|^(1/4) (fp16-operand kernel; c != 0):
    // Z <- aZ + sigma H (H + sigma b' I) Z with H = Z Z^T, b' = b / sqrt|c|.
    float zscale;    // |c|^(1/4) (1 when c == 0)
    float unscale;   // 1 / zscale
    float bq;        // sigma * b' (c != 0) or b (c == 0)
    float sigma;     // sign(c), 0 when c == 0
    // The same step with the square completed (c != 0): with the shifted
    // Gram matrix M = H + (sigma b' / 2) I, a I + P = sigma M^2 + a' I and
    // a' = a - b^2 / (4c).
    float hshift;    // sigma b' / 2 (0 when c == 0)
    float am;        // a' (a when c == 0)
    MatDesc inline_descs[kInlineMats];
    OptDesc inline_odescs[kInlineMats];
};

// Enqueue one chunk on `stream`. Returns hipErrorInvalidValue for a
// (T, storage, operand) triple without a kernel.
hipError_t launch_ns_tiled(int T, Storage st, Operand op, const KernelArgs& args, hipStream_t stream);

// True when a kernel exists for the triple (no HIP call).
bool has_kernel(int T, Storage st, Operand op);

// True when the optimizer step can run inside the tile kernel for this
// tile size, storage, operand type and sign of c (no HIP call).
bool has_step_kernel(int T, Storage st, Operand op, float c);

// The plan, descriptor upload and chunk launches of himuon_ns_tiled; with
// `opt_host` (one OptDesc per matrix) and the step's scalars, the fused
// optimizer step (has_step_kernel must hold). Returns a himuon status.
int run_tiled(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, const int64_t* rows,
              const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int T, int K, float a, float b,
              float c, int dtype, int compute, void* workspace, size_t workspace_bytes, size_t chunk_budget_bytes,
              void* stream, const OptDesc* opt_host, float beta, float decay, float lr, int nesterov);
// Workspace of run_tiled: the MatDesc table, and the OptDesc table for a step.
size_t tiled_workspace(int64_t n_mats, bool step);

// The pieces of run_tiled, shared with the entry point that allocates
// nothing. validate_tiled checks every argument of a himuon_ns_tiled call
// (no HIP call) and resolves its operand type into *op; plan_tiled_chunks
// gives the call's tile and chunk counts; make_desc builds one matrix's
// descriptor (tile_begin: its first global tile id; mom: the step's momentum
// pointer or null); make_kernel_args sets the scalars of a launch;
// launch_chunks enqueues one launch per chunk; stream_device makes the
// stream's device current (*cur: the previous one, to restore).
// Tile shapes are Th x Tw (square: Th = Tw = T); validate_tiled checks
// argument values only (the caller checks that a kernel serves the shape).
int validate_tiled(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, const int64_t* rows,
                   const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int Tw, int K, float a, float b,
                   float c, int dtype, int compute, int* op);
int plan_tiled_chunks(int64_t n_mats, const int64_t* rows, const int64_t* cols, int Th, int Tw, int dtype,
                      size_t chunk_budget_bytes, int64_t* total, int64_t* n_chunks);
MatDesc make_desc(const void* in, void* out, int64_t rows, int64_t cols, int64_t ld_in, int64_t ld_out,
                  int64_t tile_begin, int Tw, int dtype, const void* mom);
KernelArgs make_kernel_args(const MatDesc* descs, int64_t n_mats, int K, float a, float b, float c);
// Copies the tables of a call of at most kInlineMats matrices into the
// arguments (descs, odescs become null; `opt` may be null).
void set_inline_tables(KernelArgs& ka, const MatDesc* descs, const OptDesc* opt, int64_t n_mats);
int launch_chunks(int T, Storage st, Operand op, KernelArgs ka, int64_t total, int64_t n_chunks, hipStream_t stream);
int stream_device(hipStream_t stream, int* cur, int* dev);

// The fp16-operand kernel family (bf16 storage), T in {32, 64, 128, 256}.
hipError_t launch_ns_tiled_f16(int T, const KernelArgs& args, hipStream_t stream);

// The fused rectangular-tile family (ns_rect.hip): Th x Tw tiles with
// {min, max} in {32} x {64, 128, 256} (fp32 storage with fp32 operands,
// bf16 storage with fp16 or bf16 operands) or {32} x {512}, {64} x {128,
// 256} (bf16 storage only).
bool has_rect_kernel(int Th, int Tw, Storage st, Operand op);
hipError_t launch_ns_rect(int Th, int Tw, Storage st, Operand op, const KernelArgs& args, hipStream_t stream);

// Host helpers shared by the entry points (himuon_api.cpp).
extern thread_local int g_last_hip_error;
// Records `e` as the calling thread's last HIP error; returns HIMUON_ERR_HIP.
int set_hip_error(hipError_t e);
// Copies `bytes` of host data to device memory `dst` on `stream` through a
// ring of pinned staging slots (asynchronous; a slot is reused once its
// copy has completed). Returns a himuon status. While a plan is recorded on
// the calling thread (g_recording), each table gets a pinned buffer of the
// plan's own instead, which the recorded copy reads at every replay.
int upload_table(const void* data, size_t bytes, void* dst, hipStream_t stream, int dev);

// The host side of a plan being recorded (himuon_plan.cpp).
struct PlanRecording {
    std::vector<void*> host_buffers;  // pinned, freed with the plan
};
extern thread_local PlanRecording* g_recording;

// Creates the GEMM library's handle on device `dev` if it does not exist yet
// (plans create it before recording). Returns a himuon status.
int gemm_handle_ready(int dev);
// Largest |p^k(s)| over s in [0, 1], k < K, p(s) = a s + b s^3 + c s^5.
double iterate_bound(int K, double a, double b, double c);

}  // namespace himuon
