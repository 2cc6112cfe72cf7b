// C ABI of the tiled Newton–Schulz library: argument validation, the tile
// and chunk plan, descriptor upload, and one kernel launch per chunk.
//
// Plan (Sec. 4.4.2, "cross-layer batching" with memory-bounded chunking;
// Sec. 4.4.3, "runtime tile-size reconfiguration"): every matrix of a call
// contributes its R x C tiles to one global, densely numbered tile set; the
// set is split into the fewest chunks whose staged bytes fit the budget,
// balanced to within one tile. The plan is O(#matrices) integer work and is
// rebuilt on every call, so changing T between calls costs nothing extra.
#include "himuon_internal.h"
#include "ns_gemm_path.h"
#include "../../include/himuon.h"

#include <math.h>
#include <mutex>
#include <string.h>
#include <vector>

namespace {

using himuon::MatDesc;

constexpr int kVersion = 100;  // 0.1.0

size_t elem_size(int dtype) { return dtype == HIMUON_BF16 ? 2 : 4; }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Tiles per matrix prefix and total for Th x Tw tiles; validates shapes.
// Th, Tw >= 1.
int plan_tiles(int64_t n_mats, const int64_t* rows, const int64_t* cols, int64_t Th, int64_t Tw,
               std::vector<int64_t>* begin, int64_t* total)
{
    if (n_mats < 1 || !rows || !cols || Th < 1 || Tw < 1) return HIMUON_ERR_INVALID_ARG;
    int64_t acc = 0;
    if (begin) begin->resize((size_t)n_mats);
    for (int64_t m = 0; m < n_mats; ++m) {
        if (rows[m] < 1 || cols[m] < 1) return HIMUON_ERR_INVALID_ARG;
        const int64_t t = ceil_div(rows[m], Th) * ceil_div(cols[m], Tw);
        if (begin) (*begin)[(size_t)m] = acc;
        if (acc > INT64_MAX - t) return HIMUON_ERR_INVALID_ARG;
        acc += t;
    }
    *total = acc;
    return HIMUON_OK;
}

// Fewest chunks whose per-chunk bytes (2*Th*Tw*elem per tile) fit `budget`.
int plan_chunk_count(int64_t total, int64_t Th, int64_t Tw, size_t elem, size_t budget, int64_t* n_chunks)
{
    if (budget == 0) {
        *n_chunks = 1;
        return HIMUON_OK;
    }
    const unsigned __int128 per_tile = (unsigned __int128)2 * (unsigned __int128)Th * (unsigned __int128)Tw * elem;
    const unsigned __int128 fit = (unsigned __int128)budget / per_tile;
    if (fit == 0) return HIMUON_ERR_WORKSPACE;
    const int64_t per_chunk = fit > (unsigned __int128)total ? total : (int64_t)fit;
    *n_chunks = ceil_div(total, per_chunk);
    return HIMUON_OK;
}

int64_t chunk_bound(int64_t i, int64_t total, int64_t n_chunks)
{
    return (int64_t)(((__int128)i * total) / n_chunks);
}

bool finite3(float a, float b, float c) { return isfinite(a) && isfinite(b) && isfinite(c); }

int resolve_compute(int dtype, int compute, int K, float a, float b, float c)
{
    if (dtype != HIMUON_F32 && dtype != HIMUON_BF16) return HIMUON_ERR_INVALID_ARG;
    if (compute < HIMUON_COMPUTE_DEFAULT || compute > HIMUON_COMPUTE_BF16) return HIMUON_ERR_INVALID_ARG;
    if (!finite3(a, b, c) || K < 0) return HIMUON_ERR_INVALID_ARG;
    if (dtype == HIMUON_F32) {
        if (compute == HIMUON_COMPUTE_DEFAULT || compute == HIMUON_COMPUTE_F32) return HIMUON_COMPUTE_F32;
        return HIMUON_ERR_UNSUPPORTED;
    }
    if (compute == HIMUON_COMPUTE_F32) return HIMUON_ERR_UNSUPPORTED;
    if (compute == HIMUON_COMPUTE_BF16) return HIMUON_COMPUTE_BF16;
    // fp16 operands (kernel state Z = X |c|^(1/4), H = Z Z^T): Z, H,
    // H + sigma b' I, the step operator a I + sigma H (H + sigma b' I), and
    // the 256-tile chain operand Y = sigma (H + sigma b' I) Z must stay far
    // below 65504, and so must the bf16-operand path's A = X X^T and
    // B = bA + cA^2. Entries are bounded by spectral norms.
    const double M = 4.0 * himuon::iterate_bound(K, a, b, c);
    const double zs = c != 0.f ? pow(fabs((double)c), 0.25) : 1.0;
    const double bp = c != 0.f ? fabs((double)b) / sqrt(fabs((double)c)) : fabs((double)b);
    const double Mz = M * zs, MH = Mz * Mz;
    const double M2 = M * M;
    const double fp16_ops = fmax(fmax(Mz, MH + bp), fmax(fabs((double)a) + bp * MH + MH * MH, (MH + bp) * Mz));
    const double bound = fmax(fp16_ops, fmax(M2, fabs((double)b) * M2 + fabs((double)c) * M2 * M2));
    // DEFAULT never switches to bf16 operands on its own: one-pass bf16
    // operands miss the 2e-2 bf16-storage bar at T <= 64 and at K = 8, so a
    // caller who accepts that accuracy asks for HIMUON_COMPUTE_BF16.
    return bound < 16384.0 ? HIMUON_COMPUTE_F16 : HIMUON_ERR_RANGE;
}

}  // namespace

namespace himuon {

thread_local int g_last_hip_error = 0;

int set_hip_error(hipError_t e)
{
    g_last_hip_error = (int)e;
    return HIMUON_ERR_HIP;
}

// Largest |p^k(s)| over s in [0, 1] and k < K, for p(s) = a s + b s^3 + c s^5:
// each singular value of the normalised tile starts in [0, 1] and follows p
// exactly, so this bounds every entry of the operand X at every step. The
// interval is sampled densely; a factor of 4 covers what falls between points.
double iterate_bound_uncached(int K, double a, double b, double c);

// (8193 samples times K: tens of microseconds, so the last few results are
// kept; a call with the same K and coefficients reuses them.)
double iterate_bound(int K, double a, double b, double c)
{
    struct Entry {
        int K;
        double a, b, c, bound;
    };
    static std::mutex mu;
    static Entry cache[8];
    static int n_cached = 0, next_slot = 0;
    {
        std::lock_guard<std::mutex> lock(mu);
        for (int i = 0; i < n_cached; ++i)
            if (cache[i].K == K && cache[i].a == a && cache[i].b == b && cache[i].c == c) return cache[i].bound;
    }
    const double bound = iterate_bound_uncached(K, a, b, c);
    std::lock_guard<std::mutex> lock(mu);
    cache[next_slot] = Entry{K, a, b, c, bound};
    next_slot = (next_slot + 1) % 8;
    if (n_cached < 8) ++n_cached;
    return bound;
}

double iterate_bound_uncached(int K, double a, double b, double c)
{
    constexpr int kPts = 8193;
    double m = 1.0;
    for (int i = 0; i < kPts; ++i) {
        double x = (double)i / (kPts - 1);
        for (int k = 1; k < K; ++k) {
            x = a * x + b * x * x * x + c * x * x * x * x * x;
            const double ax = fabs(x);
            if (!(ax < 1e30)) return INFINITY;
            if (ax > m) m = ax;
        }
    }
    return m;
}

// Pinned host staging for the descriptor table. A ring of slots lets the
// host run several calls ahead of the GPU; a slot is reused only after the
// copy that read it has completed (its event).
struct StagingSlot {
    void* host = nullptr;
    size_t cap = 0;
    hipEvent_t ev = nullptr;
    int dev = -1;
    bool pending = false;
};

constexpr int kSlots = 8;
std::mutex g_staging_mu;
StagingSlot g_slots[kSlots];
unsigned g_next_slot = 0;

thread_local PlanRecording* g_recording = nullptr;

int upload_table(const void* data, size_t bytes, void* workspace, hipStream_t stream, int dev)
{
    if (g_recording) {
        // A plan being recorded: the table goes into a pinned buffer that the
        // plan owns, so the captured copy reads the same bytes at every replay.
        void* host = nullptr;
        hipError_t e = hipHostMalloc(&host, bytes, hipHostMallocDefault);
        if (e != hipSuccess) return set_hip_error(e);
        g_recording->host_buffers.push_back(host);
        memcpy(host, data, bytes);
        e = hipMemcpyAsync(workspace, host, bytes, hipMemcpyHostToDevice, stream);
        return e == hipSuccess ? HIMUON_OK : set_hip_error(e);
    }
    std::lock_guard<std::mutex> lock(g_staging_mu);
    StagingSlot& sl = g_slots[g_next_slot++ % kSlots];
    hipError_t e;
    if (sl.pending) {
        e = hipEventSynchronize(sl.ev);
        if (e != hipSuccess) return set_hip_error(e);
        sl.pending = false;
    }
    if (sl.cap < bytes) {
        if (sl.host) {
            e = hipHostFree(sl.host);
            if (e != hipSuccess) return set_hip_error(e);
            sl.host = nullptr;
            sl.cap = 0;
        }
        size_t cap = 4096;
        while (cap < bytes) cap *= 2;
        e = hipHostMalloc(&sl.host, cap, hipHostMallocDefault);
        if (e != hipSuccess) return set_hip_error(e);
        sl.cap = cap;
    }
    if (sl.dev != dev) {
        if (sl.ev) (void)hipEventDestroy(sl.ev);
        sl.ev = nullptr;
        e = hipEventCreateWithFlags(&sl.ev, hipEventDisableTiming);
        if (e != hipSuccess) return set_hip_error(e);
        sl.dev = dev;
    }
    memcpy(sl.host, data, bytes);
    e = hipMemcpyAsync(workspace, sl.host, bytes, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return set_hip_error(e);
    e = hipEventRecord(sl.ev, stream);
    if (e != hipSuccess) return set_hip_error(e);
    sl.pending = true;
    return HIMUON_OK;
}

}  // namespace himuon

extern "C" {

size_t himuon_ns_tiled_workspace_size(int64_t n_mats) { return himuon::tiled_workspace(n_mats, false); }

size_t himuon_ns_tiled_call_workspace_size(int64_t n_mats, const int64_t* rows, const int64_t* cols, int T, int dtype,
                                           int compute, int K, float a, float b, float c, size_t chunk_budget_bytes)
{
    if (n_mats < 1 || !rows || !cols) return 0;
    if (T != 32 && T != 64 && T != 128 && T != 256) return 0;
    const int op = resolve_compute(dtype, compute, K, a, b, c);
    if (op < 0) return 0;
    for (int64_t m = 0; m < n_mats; ++m)
        if (rows[m] < 1 || cols[m] < 1) return 0;
    const himuon::Storage st = dtype == HIMUON_BF16 ? himuon::Storage::BF16 : himuon::Storage::F32;
    if (himuon::has_kernel(T, st, (himuon::Operand)op)) return himuon::tiled_workspace(n_mats, false);
    return himuon::gemm_path_workspace(n_mats, rows, cols, T, T, dtype, op, K, a, b, c, chunk_budget_bytes);
}

int himuon_plan_chunks(int64_t n_mats, const int64_t* rows, const int64_t* cols, int T, int dtype,
                       size_t chunk_budget_bytes, int64_t* total_tiles, int64_t* n_chunks,
                       int64_t* chunk_bounds, int64_t max_bounds)
{
    if (!total_tiles || !n_chunks) return HIMUON_ERR_INVALID_ARG;
    if (dtype != HIMUON_F32 && dtype != HIMUON_BF16) return HIMUON_ERR_INVALID_ARG;
    int64_t total = 0, nc = 0;
    int st = plan_tiles(n_mats, rows, cols, T, T, nullptr, &total);
    if (st != HIMUON_OK) return st;
    st = plan_chunk_count(total, T, T, elem_size(dtype), chunk_budget_bytes, &nc);
    if (st != HIMUON_OK) return st;
    *total_tiles = total;
    *n_chunks = nc;
    if (chunk_bounds && max_bounds >= nc + 1)
        for (int64_t i = 0; i <= nc; ++i) chunk_bounds[i] = chunk_bound(i, total, nc);
    return HIMUON_OK;
}

int himuon_select_compute(int dtype, int compute, int K, float a, float b, float c)
{
    return resolve_compute(dtype, compute, K, a, b, c);
}

}  // extern "C"

namespace himuon {

size_t tiled_workspace(int64_t n_mats, bool step)
{
    if (n_mats < 1) return 0;
    const size_t b = (size_t)n_mats * sizeof(MatDesc);
    const size_t o = step ? (size_t)n_mats * sizeof(OptDesc) : 0;
    return (b + 255) / 256 * 256 + (o + 255) / 256 * 256;
}

bool has_step_kernel(int T, Storage st, Operand op, float c)
{
    if (T != 32 && T != 64 && T != 128) return false;
    if (op == Operand::F16) return st == Storage::BF16 && c > 0.f;  // the fp16 kernels' step variants
    return has_kernel(T, st, op);                                   // fp32 storage, bf16 operands
}

int validate_tiled(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, const int64_t* rows,
                   const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int Tw, int K, float a, float b,
                   float c, int dtype, int compute, int* op)
{
    if (n_mats < 1 || n_mats > INT32_MAX || !in_ptrs || !out_ptrs || !rows || !cols) return HIMUON_ERR_INVALID_ARG;
    if (K < 0 || !finite3(a, b, c)) return HIMUON_ERR_INVALID_ARG;
    if (dtype != HIMUON_F32 && dtype != HIMUON_BF16) return HIMUON_ERR_INVALID_ARG;
    if (compute < HIMUON_COMPUTE_DEFAULT || compute > HIMUON_COMPUTE_BF16) return HIMUON_ERR_INVALID_ARG;
    if (Tw < 1) return HIMUON_ERR_UNSUPPORTED;
    for (int64_t m = 0; m < n_mats; ++m) {
        if (!in_ptrs[m] || !out_ptrs[m] || rows[m] < 1 || cols[m] < 1) return HIMUON_ERR_INVALID_ARG;
        const int64_t li = ld_in ? ld_in[m] : cols[m];
        const int64_t lo = ld_out ? ld_out[m] : cols[m];
        if (li < cols[m] || lo < cols[m]) return HIMUON_ERR_INVALID_ARG;
        if (rows[m] > INT64_MAX / li || rows[m] > INT64_MAX / lo) return HIMUON_ERR_INVALID_ARG;
        if (ceil_div(cols[m], Tw) > INT32_MAX) return HIMUON_ERR_INVALID_ARG;
    }
    const int r = resolve_compute(dtype, compute, K, a, b, c);
    if (r < 0) return r;
    *op = r;
    return HIMUON_OK;
}

int plan_tiled_chunks(int64_t n_mats, const int64_t* rows, const int64_t* cols, int Th, int Tw, int dtype,
                      size_t chunk_budget_bytes, int64_t* total, int64_t* n_chunks)
{
    int s = plan_tiles(n_mats, rows, cols, Th, Tw, nullptr, total);
    if (s != HIMUON_OK) return s;
    s = plan_chunk_count(*total, Th, Tw, elem_size(dtype), chunk_budget_bytes, n_chunks);
    if (s != HIMUON_OK) return s;
    // the kernels number the tiles of a call with 32-bit ids
    if (*total > (int64_t)UINT32_MAX) return HIMUON_ERR_UNSUPPORTED;
    return HIMUON_OK;
}

MatDesc make_desc(const void* in, void* out, int64_t rows, int64_t cols, int64_t ld_in, int64_t ld_out,
                  int64_t tile_begin, int Tw, int dtype, const void* mom)
{
    // 16-byte accesses at every column multiple of 8 (bf16) or 4 (f32)
    const size_t align = 16;
    const int64_t ld_mult = dtype == HIMUON_BF16 ? 8 : 4;
    MatDesc d;
    d.in = in;
    d.out = out;
    d.rows = rows;
    d.cols = cols;
    d.ld_in = ld_in;
    d.ld_out = ld_out;
    d.tile_begin = tile_begin;
    d.tiles_c = (int32_t)ceil_div(cols, Tw);
    d.flags = 0;
    // (a step's momentum shares the gradient's layout and alignment flag)
    if ((uintptr_t)in % align == 0 && ld_in % ld_mult == 0 && (!mom || (uintptr_t)mom % align == 0))
        d.flags |= MAT_VEC_IN;
    if ((uintptr_t)out % align == 0 && ld_out % ld_mult == 0) d.flags |= MAT_VEC_OUT;
    return d;
}

KernelArgs make_kernel_args(const MatDesc* descs, int64_t n_mats, int K, float a, float b, float c)
{
    KernelArgs ka{};
    ka.descs = descs;
    ka.odescs = nullptr;
    ka.step = 0;
    ka.beta = 0.f;
    ka.decay = 1.f;
    ka.lr = 0.f;
    ka.nesterov = 0;
    ka.n_mats = (int32_t)n_mats;
    ka.K = K;
    ka.a = a;
    ka.b = b;
    ka.c = c;
    ka.b_over_c = c != 0.f ? b / c : 0.f;
    if (c != 0.f) {
        const double ac = fabs((double)c);
        ka.zscale = (float)pow(ac, 0.25);
        ka.unscale = (float)(1.0 / pow(ac, 0.25));
        ka.sigma = c > 0.f ? 1.f : -1.f;
        ka.bq = (float)((double)ka.sigma * (double)b / sqrt(ac));
        ka.hshift = (float)(0.5 * (double)ka.sigma * (double)b / sqrt(ac));
        ka.am = (float)((double)a - (double)b * (double)b / (4.0 * (double)c));
    } else {
        ka.zscale = 1.f;
        ka.unscale = 1.f;
        ka.sigma = 0.f;
        ka.bq = b;
        ka.hshift = 0.f;
        ka.am = a;
    }
    return ka;
}

void set_inline_tables(KernelArgs& ka, const MatDesc* descs, const OptDesc* opt, int64_t n_mats)
{
    ka.descs = nullptr;
    ka.odescs = nullptr;
    for (int64_t m = 0; m < n_mats; ++m) {
        ka.inline_descs[m] = descs[m];
        if (opt) ka.inline_odescs[m] = opt[m];
    }
}

int launch_chunks(int T, Storage st, Operand op, KernelArgs ka, int64_t total, int64_t n_chunks, hipStream_t stream)
{
    for (int64_t i = 0; i < n_chunks; ++i) {
        ka.tile_begin = chunk_bound(i, total, n_chunks);
        ka.tile_end = chunk_bound(i + 1, total, n_chunks);
        const hipError_t e = launch_ns_tiled(T, st, op, ka, stream);
        if (e != hipSuccess) return set_hip_error(e);
    }
    return HIMUON_OK;
}

int stream_device(hipStream_t stream, int* cur, int* dev)
{
    hipError_t e = hipGetDevice(cur);
    if (e != hipSuccess) return set_hip_error(e);
    *dev = *cur;
    if (stream) {
        e = hipStreamGetDevice(stream, dev);
        if (e != hipSuccess) return set_hip_error(e);
    }
    if (*dev != *cur && (e = hipSetDevice(*dev)) != hipSuccess) return set_hip_error(e);
    return HIMUON_OK;
}

int run_tiled(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, const int64_t* rows,
              const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int T, int K, float a, float b,
              float c, int dtype, int compute, void* workspace, size_t workspace_bytes, size_t chunk_budget_bytes,
              void* stream, const OptDesc* opt_host, float beta, float decay, float lr, int nesterov)
{
    // ---- validation: nothing is enqueued unless every check passes
    int op = 0;
    if (T != 32 && T != 64 && T != 128 && T != 256) {
        const int s = validate_tiled(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, 32, K, a, b, c, dtype,
                                     compute, &op);
        return s != HIMUON_OK ? s : HIMUON_ERR_UNSUPPORTED;
    }
    int s = validate_tiled(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, T, K, a, b, c, dtype, compute, &op);
    if (s != HIMUON_OK) return s;
    const Storage st = dtype == HIMUON_BF16 ? Storage::BF16 : Storage::F32;
    const Operand opnd = (Operand)op;
    if (!has_kernel(T, st, opnd)) {
        // 256-tiles without a fused kernel (fp32 storage, bf16 operands): each
        // tile is a 256 x 256 problem of the library-GEMM path, in the same call
        if (T == 256 && !opt_host)
            return run_gemm_path(n_mats, in_ptrs, out_ptrs, nullptr, nullptr, rows, cols, ld_in, ld_out, T, T, K, a,
                                 b, c, dtype, op, workspace, workspace_bytes, chunk_budget_bytes, stream, nullptr);
        return HIMUON_ERR_UNSUPPORTED;
    }
    if (opt_host && !has_step_kernel(T, st, opnd, c)) return HIMUON_ERR_UNSUPPORTED;
    if (!workspace || workspace_bytes < tiled_workspace(n_mats, opt_host != nullptr)) return HIMUON_ERR_WORKSPACE;
    int64_t total = 0, n_chunks = 0;
    s = plan_tiled_chunks(n_mats, rows, cols, T, T, dtype, chunk_budget_bytes, &total, &n_chunks);
    if (s != HIMUON_OK) return s;

    // ---- descriptor table
    std::vector<MatDesc> descs((size_t)n_mats);
    int64_t next = 0;
    for (int64_t m = 0; m < n_mats; ++m) {
        descs[(size_t)m] = make_desc(in_ptrs[m], out_ptrs[m], rows[m], cols[m], ld_in ? ld_in[m] : cols[m],
                                     ld_out ? ld_out[m] : cols[m], next, T, dtype,
                                     opt_host ? opt_host[m].mom : nullptr);
        next += ceil_div(rows[m], T) * ceil_div(cols[m], T);
    }

    // ---- run on the stream's device
    hipStream_t hs = static_cast<hipStream_t>(stream);
    int cur = 0, dev = 0;
    s = stream_device(hs, &cur, &dev);
    if (s != HIMUON_OK) return s;
    const size_t dbytes = ((size_t)n_mats * sizeof(MatDesc) + 255) / 256 * 256;
    OptDesc* const otab = opt_host ? reinterpret_cast<OptDesc*>(static_cast<uint8_t*>(workspace) + dbytes) : nullptr;
    // A call of few matrices carries its tables in the launch arguments;
    // larger ones copy them into the workspace ahead of the kernels.
    const bool inl = n_mats <= kInlineMats;
    int status = HIMUON_OK;
    if (!inl) {
        status = upload_table(descs.data(), descs.size() * sizeof(MatDesc), workspace, hs, dev);
        if (status == HIMUON_OK && opt_host)
            status = upload_table(opt_host, (size_t)n_mats * sizeof(OptDesc), otab, hs, dev);
    }
    if (status == HIMUON_OK) {
        KernelArgs ka = make_kernel_args(static_cast<const MatDesc*>(workspace), n_mats, K, a, b, c);
        ka.odescs = otab;
        ka.step = opt_host ? 1 : 0;
        if (inl) set_inline_tables(ka, descs.data(), opt_host, n_mats);
        ka.beta = beta;
        ka.decay = decay;
        ka.lr = lr;
        ka.nesterov = nesterov;
        status = launch_chunks(T, st, opnd, ka, total, n_chunks, hs);
    }
    if (dev != cur) (void)hipSetDevice(cur);
    return status;
}

int run_tiled_hw(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, const int64_t* rows,
                 const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int Th, int Tw, int K, float a,
                 float b, float c, int dtype, int compute, void* workspace, size_t workspace_bytes,
                 size_t chunk_budget_bytes, void* stream)
{
    int op = 0;
    int s = validate_tiled(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, Tw < 1 ? 1 : Tw, K, a, b, c,
                           dtype, compute, &op);
    if (s != HIMUON_OK) return s;
    if (Th < 1 || Tw < 1) return HIMUON_ERR_INVALID_ARG;
    const Storage st = dtype == HIMUON_BF16 ? Storage::BF16 : Storage::F32;
    const Operand opnd = (Operand)op;
    if (!has_rect_kernel(Th, Tw, st, opnd)) return HIMUON_ERR_UNSUPPORTED;
    if (!workspace || workspace_bytes < tiled_workspace(n_mats, false)) return HIMUON_ERR_WORKSPACE;
    int64_t total = 0, n_chunks = 0;
    s = plan_tiled_chunks(n_mats, rows, cols, Th, Tw, dtype, chunk_budget_bytes, &total, &n_chunks);
    if (s != HIMUON_OK) return s;

    std::vector<MatDesc> descs((size_t)n_mats);
    int64_t next = 0;
    for (int64_t m = 0; m < n_mats; ++m) {
        descs[(size_t)m] = make_desc(in_ptrs[m], out_ptrs[m], rows[m], cols[m], ld_in ? ld_in[m] : cols[m],
                                     ld_out ? ld_out[m] : cols[m], next, Tw, dtype, nullptr);
        next += ceil_div(rows[m], Th) * ceil_div(cols[m], Tw);
    }
    hipStream_t hs = static_cast<hipStream_t>(stream);
    int cur = 0, dev = 0;
    s = stream_device(hs, &cur, &dev);
    if (s != HIMUON_OK) return s;
    const bool inl = n_mats <= kInlineMats;
    int status = inl ? HIMUON_OK : upload_table(descs.data(), descs.size() * sizeof(MatDesc), workspace, hs, dev);
    if (status == HIMUON_OK) {
        KernelArgs ka = make_kernel_args(static_cast<const MatDesc*>(workspace), n_mats, K, a, b, c);
        if (inl) set_inline_tables(ka, descs.data(), nullptr, n_mats);
        for (int64_t i = 0; i < n_chunks && status == HIMUON_OK; ++i) {
            ka.tile_begin = chunk_bound(i, total, n_chunks);
            ka.tile_end = chunk_bound(i + 1, total, n_chunks);
            const hipError_t e = launch_ns_rect(Th, Tw, st, opnd, ka, hs);
            if (e != hipSuccess) status = set_hip_error(e);
        }
    }
    if (dev != cur) (void)hipSetDevice(cur);
    return status;
}

}  // namespace himuon

extern "C" {

int himuon_ns_tiled_hw(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, const int64_t* rows,
                       const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int Th, int Tw, int K,
                       float a, float b, float c, int dtype, int compute, void* workspace, size_t workspace_bytes,
                       size_t chunk_budget_bytes, void* stream)
{
    if (Th == Tw)
        return himuon::run_tiled(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, Th, K, a, b, c, dtype,
                                 compute, workspace, workspace_bytes, chunk_budget_bytes, stream, nullptr, 0.f, 1.f,
                                 0.f, 0);
    return himuon::run_tiled_hw(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, Th, Tw, K, a, b, c, dtype,
                                compute, workspace, workspace_bytes, chunk_budget_bytes, stream);
}

int himuon_ns_tiled(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, const int64_t* rows,
                    const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int T, int K, float a,
                    float b, float c, int dtype, int compute, void* workspace, size_t workspace_bytes,
                    size_t chunk_budget_bytes, void* stream)
{
    return himuon::run_tiled(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, T, K, a, b, c, dtype, compute,
                             workspace, workspace_bytes, chunk_budget_bytes, stream, nullptr, 0.f, 1.f, 0.f, 0);
}

const char* himuon_status_string(int status)
{
    switch (status) {
    case HIMUON_OK: return "success";
    case HIMUON_ERR_INVALID_ARG: return "invalid argument";
    case HIMUON_ERR_UNSUPPORTED: return "unsupported tile size or dtype/compute combination";
    case HIMUON_ERR_WORKSPACE: return "workspace or chunk budget too small";
    case HIMUON_ERR_HIP: return "HIP runtime error";
    case HIMUON_ERR_RANGE: return "fp16 operands would leave the fp16 range for these coefficients";
    default: return "unknown status";
    }
}

int himuon_last_hip_error(void) { return himuon::g_last_hip_error; }

int himuon_version(void) { return kVersion; }

}  // extern "C"
