// The library-GEMM path: Phi_K of whole matrices (T = 0, the full-matrix
// branch, Sec. 4.4.3) and of large tiles (T >= 1, e.g. 512, which cannot
// stay on one CU; Sec. 4.4.1's multi-kernel path), batched over problems of
// equal shape (Sec. 4.4.2).
//
// A problem is an h x w block worked on as an m x n iterate with m <= n
// (ns_gemm_path.h). Per step of eq. (ns_iteration), on a batch of iterates
// stored row-major with stride m*n:
//     A = X X^T                       (m x m, one GEMM)
//     B = (c / s^4) A A + (b / s^2) A (one GEMM, C = A)
//     X <- B X + a X                  (one GEMM, C = X)
// X is the rescaled iterate s * X_true: s^2 = min(m, 4096) for fp16 operands,
// which lifts the O(1/sqrt(mn)) entries of X off fp16's subnormal range and
// keeps X, A = s^2 A_true and B = b A_true + c A_true^2 inside its range for
// every m when the scalar iterates stay below the bound checked at planning
// (himuon_select_compute's argument, on |X|, |A| and |B|); s = 1 for fp32 and
// bf16 operands. Accumulation is fp32 in every
// mode. The GEMMs are hipBLASLt's (column-major: a row-major m x n iterate
// is an n x m column-major matrix, and A and B are symmetric).
#include "ns_gemm_path.h"
#include "himuon_internal.h"
#include "../../include/himuon.h"

#include <hipblaslt/hipblaslt.h>

#include <map>
#include <math.h>
#include <mutex>
#include <tuple>
#include <vector>

namespace {

using himuon::GemmOperand;
using himuon::GemmProb;
using himuon::GemmStore;

constexpr size_t kAlign = 256;
constexpr size_t kLtWorkspace = size_t(64) << 20;  // hipBLASLt scratch, carved from the caller's workspace
constexpr int kMaxChunkProbs = 65535;               // grid y of the gather / scatter kernels
constexpr int kMaxDevices = 64;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

size_t op_size(GemmOperand op) { return op == GemmOperand::F32 ? 4 : 2; }

hipDataType op_type(GemmOperand op)
{
    return op == GemmOperand::F32 ? HIP_R_32F : (op == GemmOperand::F16 ? HIP_R_16F : HIP_R_16BF);
}

// ---- shapes and chunks

struct Group {
    int m = 0, n = 0;      // iterate shape
    int nparts = 1;        // norm partials per problem
    int64_t count = 0;     // problems
    int64_t first = 0;     // index of the group's first problem in the call's table
    int64_t cap = 0;       // problems per chunk
    int64_t n_chunks = 0;
    size_t bytes_pp = 0;   // iterate buffers per problem (X, X', A, B)
};

int group_nparts(int n) { return (int)std::min<int64_t>(256, std::max<int64_t>(1, ceil_div(n, 64))); }

// Tiles are Th x Tw (square: Th = Tw = T; rectangular tiles are the
// tile-shape study's); Th = Tw = 0 stands for T = infinity. A matrix is one
// whole problem on that branch or when one tile covers it (Th >= H and
// Tw >= W): the tiling operator then gives a single padded tile, and Phi_K
// of a zero-padded matrix is the padded Phi_K of the matrix (Sec. 4.4.3), so
// the smaller unpadded problem is worked on instead.
bool whole_matrix(int64_t rows, int64_t cols, int Th, int Tw) { return Th == 0 || (Th >= rows && Tw >= cols); }

bool valid_tiling(int Th, int Tw) { return Th >= 0 && Tw >= 0 && (Th == 0) == (Tw == 0); }

// Groups (in order of first appearance) and, when `probs` is given, the
// problem list in group order. Whole matrices: one problem each; otherwise
// the R x C tiles of the matrix, row-major.
int plan_groups(int64_t n_mats, const int64_t* rows, const int64_t* cols, int Th, int Tw, std::vector<Group>& groups,
                std::vector<std::vector<int64_t>>* members)
{
    if (n_mats < 1 || !rows || !cols || !valid_tiling(Th, Tw)) return HIMUON_ERR_INVALID_ARG;
    groups.clear();
    std::map<std::pair<int, int>, size_t> index;
    std::vector<std::vector<int64_t>> mem;
    for (int64_t l = 0; l < n_mats; ++l) {
        if (rows[l] < 1 || cols[l] < 1) return HIMUON_ERR_INVALID_ARG;
        int64_t m, n, cnt;
        if (whole_matrix(rows[l], cols[l], Th, Tw)) {
            m = std::min(rows[l], cols[l]);
            n = std::max(rows[l], cols[l]);
            cnt = 1;
        } else {
            m = std::min(Th, Tw);
            n = std::max(Th, Tw);
            cnt = ceil_div(rows[l], Th) * ceil_div(cols[l], Tw);
        }
        if (m > 32768 || n > INT32_MAX / 32) return HIMUON_ERR_UNSUPPORTED;
        const auto key = std::make_pair((int)m, (int)n);
        auto it = index.find(key);
        if (it == index.end()) {
            Group g;
            g.m = (int)m;
            g.n = (int)n;
            g.nparts = group_nparts((int)n);
            it = index.emplace(key, groups.size()).first;
            groups.push_back(g);
            mem.emplace_back();
        }
        groups[it->second].count += cnt;
        mem[it->second].push_back(l);
    }
    int64_t acc = 0;
    for (Group& g : groups) {
        g.first = acc;
        acc += g.count;
    }
    if (members) *members = std::move(mem);
    return HIMUON_OK;
}

// Chunk capacity per group under `budget` (0: everything in one chunk, up
// to the launch limit) and the workspace bytes the call needs.
int plan_chunks(std::vector<Group>& groups, GemmOperand op, size_t budget, size_t* ws_bytes)
{
    const size_t es = op_size(op);
    int64_t total = 0;
    size_t part_max = 0, buf_max = 0;
    for (Group& g : groups) {
        const size_t mn = (size_t)g.m * g.n, mm = (size_t)g.m * g.m;
        g.bytes_pp = (2 * mn + 2 * mm) * es;
        int64_t cap = g.count;
        if (budget) {
            const int64_t fit = (int64_t)(budget / g.bytes_pp);
            if (fit < 1) return HIMUON_ERR_WORKSPACE;
            cap = std::min<int64_t>(cap, fit);
        }
        cap = std::min<int64_t>(cap, kMaxChunkProbs);
        g.n_chunks = ceil_div(g.count, cap);
        g.cap = ceil_div(g.count, g.n_chunks);  // balanced
        total += g.count;
        part_max = std::max(part_max, (size_t)g.cap * g.nparts * sizeof(double));
        buf_max = std::max(buf_max, 2 * align_up((size_t)g.cap * mn * es) + 2 * align_up((size_t)g.cap * mm * es));
    }
    *ws_bytes = align_up((size_t)total * sizeof(GemmProb)) + align_up(part_max) + buf_max + kLtWorkspace;
    return HIMUON_OK;
}

// Square of the fp16 iterate scale for an m x n iterate (see the file comment).
double fp16_scale2(int m) { return (double)std::min(m, 4096); }

// Scale of the iterate in the GEMM buffers for operand type `op`.
double iterate_scale(GemmOperand op, int m) { return op == GemmOperand::F16 ? sqrt(fp16_scale2(m)) : 1.0; }

// fp16 operands keep s*X, s^2 A and B inside fp16 (see the file comment).
// DEFAULT takes them when that holds and otherwise fails with
// HIMUON_ERR_RANGE; bf16 operands are used only when asked for.
int resolve_operand(int dtype, int compute, int K, float a, float b, float c, int m_max, GemmOperand* op)
{
    if (dtype == HIMUON_F32) {
        if (compute != HIMUON_COMPUTE_DEFAULT && compute != HIMUON_COMPUTE_F32) return HIMUON_ERR_UNSUPPORTED;
        *op = GemmOperand::F32;
        return HIMUON_OK;
    }
    if (compute == HIMUON_COMPUTE_F32) return HIMUON_ERR_UNSUPPORTED;
    if (compute == HIMUON_COMPUTE_BF16) {
        *op = GemmOperand::BF16;
        return HIMUON_OK;
    }
    // |X| <= M, so |s X| <= M s, |s^2 A| <= M^2 s^2 and |B| <= |b| M^2 + |c| M^4
    // (M from the sampled scalar iterates, K + 1 of them: the output is an
    // operand-typed iterate too; 1.25 covers what falls between samples)
    const double M = 1.25 * himuon::iterate_bound(K + 1, a, b, c);
    const double s2 = fp16_scale2(m_max);
    const double bound = fmax(M * sqrt(s2), fmax(M * M * s2, fabs((double)b) * M * M + fabs((double)c) * M * M * M * M));
    if (!(bound < 32768.0)) return HIMUON_ERR_RANGE;
    *op = GemmOperand::F16;
    return HIMUON_OK;
}

// ---- hipBLASLt plans

std::mutex g_lt_mu;
hipblasLtHandle_t g_lt[kMaxDevices] = {};

// One host thread at a time enqueues GEMM-path work: the per-device
// hipBLASLt handle is shared by every calling thread (nothing establishes
// that concurrent hipblasLtMatmul calls on one handle are safe), and the
// tuner rewrites a plan's chosen algorithm, which a concurrent call reads.
// Held over the enqueue only (microseconds per GEMM), never over device
// work; taken before g_lt_mu where both are held.
std::mutex g_enqueue_mu;

constexpr int kCandidates = 32;  // heuristic results kept per GEMM for himuon_gemm_tune

struct Gemm {
    hipblasLtMatmulDesc_t desc = nullptr;
    hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, lc = nullptr;
    hipblasLtMatmulAlgo_t algo{};  // in use: the heuristic's first choice, or the tuned one
    hipblasLtMatmulAlgo_t cand[kCandidates];
    int n_cand = 0;
};

struct Plan {
    Gemm gram, poly, apply;  // A = X X^T; B = alpha A A + beta A; X' = X B + a X (column-major view)
    bool tuned = false;
};

std::map<std::tuple<int, int, int, int, int>, Plan> g_plans;  // (dev, m, n, batch, op)

hipblasLtMatrixLayout_t make_layout(hipDataType t, int64_t rows, int64_t cols, int64_t ld, int batch, int64_t stride)
{
    hipblasLtMatrixLayout_t l = nullptr;
    if (hipblasLtMatrixLayoutCreate(&l, t, (uint64_t)rows, (uint64_t)cols, ld) != HIPBLAS_STATUS_SUCCESS) return nullptr;
    const int32_t bc = batch;
    if (hipblasLtMatrixLayoutSetAttribute(l, HIPBLASLT_MATRIX_LAYOUT_BATCH_COUNT, &bc, sizeof(bc)) != HIPBLAS_STATUS_SUCCESS ||
        hipblasLtMatrixLayoutSetAttribute(l, HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET, &stride, sizeof(stride)) !=
            HIPBLAS_STATUS_SUCCESS) {
        hipblasLtMatrixLayoutDestroy(l);
        return nullptr;
    }
    return l;
}

bool make_gemm(hipblasLtHandle_t h, Gemm& g, hipblasOperation_t ta, hipDataType t, int64_t ar, int64_t ac, int64_t ald,
               int64_t as, int64_t br, int64_t bc, int64_t bld, int64_t bs, int64_t cr, int64_t cc, int64_t cld,
               int64_t cs, int batch)
{
    const hipblasComputeType_t ct = HIPBLAS_COMPUTE_32F;
    if (hipblasLtMatmulDescCreate(&g.desc, ct, HIP_R_32F) != HIPBLAS_STATUS_SUCCESS) return false;
    const int32_t opa = ta, opb = HIPBLAS_OP_N;
    if (hipblasLtMatmulDescSetAttribute(g.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opa, sizeof(opa)) != HIPBLAS_STATUS_SUCCESS ||
        hipblasLtMatmulDescSetAttribute(g.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opb, sizeof(opb)) != HIPBLAS_STATUS_SUCCESS)
        return false;
    g.la = make_layout(t, ar, ac, ald, batch, as);
    g.lb = make_layout(t, br, bc, bld, batch, bs);
    g.lc = make_layout(t, cr, cc, cld, batch, cs);
    if (!g.la || !g.lb || !g.lc) return false;
    hipblasLtMatmulPreference_t pref = nullptr;
    if (hipblasLtMatmulPreferenceCreate(&pref) != HIPBLAS_STATUS_SUCCESS) return false;
    const uint64_t wsmax = kLtWorkspace;
    bool ok = hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &wsmax,
                                                    sizeof(wsmax)) == HIPBLAS_STATUS_SUCCESS;
    hipblasLtMatmulHeuristicResult_t res[kCandidates];
    int found = 0;
    ok = ok && hipblasLtMatmulAlgoGetHeuristic(h, g.desc, g.la, g.lb, g.lc, g.lc, pref, kCandidates, res, &found) ==
                   HIPBLAS_STATUS_SUCCESS;
    hipblasLtMatmulPreferenceDestroy(pref);
    if (!ok) return false;
    g.n_cand = 0;
    for (int i = 0; i < found && i < kCandidates; ++i)
        if (res[i].state == HIPBLAS_STATUS_SUCCESS && res[i].workspaceSize <= kLtWorkspace) g.cand[g.n_cand++] = res[i].algo;
    if (g.n_cand < 1) return false;
    g.algo = g.cand[0];
    return true;
}

// The three GEMMs for a batch of m x n iterates (built once per shape).
int get_plan(int dev, int m, int n, int batch, GemmOperand op, hipblasLtHandle_t* handle, Plan** plan)
{
    std::lock_guard<std::mutex> lock(g_lt_mu);
    if (dev < 0 || dev >= kMaxDevices) return himuon::set_hip_error(hipErrorInvalidDevice);
    if (!g_lt[dev]) {
        if (hipblasLtCreate(&g_lt[dev]) != HIPBLAS_STATUS_SUCCESS) {
            g_lt[dev] = nullptr;
            return himuon::set_hip_error(hipErrorInitializationError);
        }
    }
    *handle = g_lt[dev];
    const auto key = std::make_tuple(dev, m, n, batch, (int)op);
    auto it = g_plans.find(key);
    if (it == g_plans.end()) {
        Plan p;
        const hipDataType t = op_type(op);
        const int64_t mn = (int64_t)m * n, mm = (int64_t)m * m;
        // A (m x m) = Xc^T Xc, Xc the n x m column-major view of X
        bool ok = make_gemm(g_lt[dev], p.gram, HIPBLAS_OP_T, t, n, m, n, mn, n, m, n, mn, m, m, m, mm, batch);
        // B = alpha A A + beta A
        ok = ok && make_gemm(g_lt[dev], p.poly, HIPBLAS_OP_N, t, m, m, m, mm, m, m, m, mm, m, m, m, mm, batch);
        // X'c (n x m) = Xc B + a Xc
        ok = ok && make_gemm(g_lt[dev], p.apply, HIPBLAS_OP_N, t, n, m, n, mn, m, m, m, mm, n, m, n, mn, batch);
        if (!ok) return HIMUON_ERR_UNSUPPORTED;
        it = g_plans.emplace(key, p).first;
    }
    *plan = &it->second;
    return HIMUON_OK;
}

int run_gemm(hipblasLtHandle_t h, const Gemm& g, float alpha, const void* A, const void* B, float beta, const void* C,
             void* D, void* lt_ws, hipStream_t stream)
{
    const hipblasStatus_t s = hipblasLtMatmul(h, g.desc, &alpha, A, g.la, B, g.lb, &beta, C, g.lc, D, g.lc, &g.algo,
                                              lt_ws, kLtWorkspace, stream);
    return s == HIPBLAS_STATUS_SUCCESS ? HIMUON_OK : himuon::set_hip_error(hipErrorLaunchFailure);
}

// Times every kept candidate of `g` on the given operands (three runs after
// one warm-up, on `stream`, synchronising) and keeps the fastest in g.algo.
int tune_gemm(hipblasLtHandle_t h, Gemm& g, float alpha, const void* A, const void* B, float beta, const void* C,
              void* D, void* lt_ws, hipStream_t stream, hipEvent_t e0, hipEvent_t e1)
{
    float best = 0.f;
    int best_i = -1;
    for (int i = 0; i < g.n_cand; ++i) {
        g.algo = g.cand[i];
        if (run_gemm(h, g, alpha, A, B, beta, C, D, lt_ws, stream) != HIMUON_OK) continue;
        if (hipEventRecord(e0, stream) != hipSuccess) return himuon::set_hip_error(hipGetLastError());
        int st = HIMUON_OK;
        for (int r = 0; r < 3 && st == HIMUON_OK; ++r) st = run_gemm(h, g, alpha, A, B, beta, C, D, lt_ws, stream);
        if (st != HIMUON_OK) continue;
        hipError_t e = hipEventRecord(e1, stream);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float ms = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
        if (e != hipSuccess) return himuon::set_hip_error(e);
        if (best_i < 0 || ms < best) {
            best = ms;
            best_i = i;
        }
    }
    g.algo = g.cand[best_i < 0 ? 0 : best_i];
    return HIMUON_OK;
}

}  // namespace

namespace himuon {

int gemm_handle_ready(int dev)
{
    std::lock_guard<std::mutex> lock(g_lt_mu);
    if (dev < 0 || dev >= kMaxDevices) return set_hip_error(hipErrorInvalidDevice);
    if (!g_lt[dev] && hipblasLtCreate(&g_lt[dev]) != HIPBLAS_STATUS_SUCCESS) {
        g_lt[dev] = nullptr;
        return set_hip_error(hipErrorInitializationError);
    }
    return HIMUON_OK;
}

int run_gemm_path(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, void* const* mom_ptrs,
                  const float* tau, const int64_t* rows, const int64_t* cols, const int64_t* ld_in,
                  const int64_t* ld_out, int Th, int Tw, int K, float a, float b, float c, int dtype, int compute,
                  void* workspace, size_t workspace_bytes, size_t chunk_budget_bytes, void* stream,
                  const OptArgs* opt)
{
    // ---- validation and plan: nothing is enqueued unless every check passes
    if (n_mats < 1 || n_mats > INT32_MAX || !in_ptrs || !out_ptrs || !rows || !cols) return HIMUON_ERR_INVALID_ARG;
    if (K < 0 || !valid_tiling(Th, Tw) || !isfinite(a) || !isfinite(b) || !isfinite(c)) return HIMUON_ERR_INVALID_ARG;
    if (dtype != HIMUON_F32 && dtype != HIMUON_BF16) return HIMUON_ERR_INVALID_ARG;
    if (compute < HIMUON_COMPUTE_DEFAULT || compute > HIMUON_COMPUTE_BF16) return HIMUON_ERR_INVALID_ARG;
    for (int64_t l = 0; l < n_mats; ++l) {
        if (!in_ptrs[l] || !out_ptrs[l] || rows[l] < 1 || cols[l] < 1) return HIMUON_ERR_INVALID_ARG;
        if (opt && (!mom_ptrs || !mom_ptrs[l] || !tau || !isfinite(tau[l]))) return HIMUON_ERR_INVALID_ARG;
        const int64_t li = ld_in ? ld_in[l] : cols[l];
        const int64_t lo = ld_out ? ld_out[l] : cols[l];
        if (li < cols[l] || lo < cols[l]) return HIMUON_ERR_INVALID_ARG;
        if (rows[l] > INT64_MAX / li || rows[l] > INT64_MAX / lo) return HIMUON_ERR_INVALID_ARG;
        if (rows[l] > INT32_MAX || cols[l] > INT32_MAX) return HIMUON_ERR_UNSUPPORTED;
    }
    std::vector<Group> groups;
    std::vector<std::vector<int64_t>> members;
    int st = plan_groups(n_mats, rows, cols, Th, Tw, groups, &members);
    if (st != HIMUON_OK) return st;
    int m_max = 0;
    for (const Group& g : groups) m_max = std::max(m_max, g.m);
    GemmOperand op;
    st = resolve_operand(dtype, compute, K, a, b, c, m_max, &op);
    if (st != HIMUON_OK) return st;
    size_t need = 0;
    st = plan_chunks(groups, op, chunk_budget_bytes, &need);
    if (st != HIMUON_OK) return st;
    if (!workspace || workspace_bytes < need) return HIMUON_ERR_WORKSPACE;
    const GemmStore sto = dtype == HIMUON_BF16 ? GemmStore::BF16 : GemmStore::F32;

    // problem table, in group order
    std::vector<GemmProb> probs;
    int64_t total = 0;
    for (const Group& g : groups) total += g.count;
    probs.reserve((size_t)total);
    for (size_t gi = 0; gi < groups.size(); ++gi) {
        for (const int64_t l : members[gi]) {
            GemmProb p{};
            p.in = in_ptrs[l];
            p.out = out_ptrs[l];
            p.ld_in = ld_in ? ld_in[l] : cols[l];
            p.ld_out = ld_out ? ld_out[l] : cols[l];
            p.mom = opt ? mom_ptrs[l] : nullptr;
            p.tau = opt ? tau[l] : 0.f;
            // 16-byte chunks at every 8th column of a block (block origins are multiples of Tw)
            const int64_t mult = dtype == HIMUON_BF16 ? 8 : 4;
            const bool origins = Tw % 8 == 0;
            const bool vin = origins && (uintptr_t)p.in % 16 == 0 && p.ld_in % mult == 0 &&
                             (!opt || (uintptr_t)p.mom % 16 == 0);
            const bool vout = origins && (uintptr_t)p.out % 16 == 0 && p.ld_out % mult == 0;
            p.vec = (vin ? himuon::GEMM_VEC_IN : 0) | (vout ? himuon::GEMM_VEC_OUT : 0);
            if (whole_matrix(rows[l], cols[l], Th, Tw)) {
                p.row0 = p.col0 = 0;
                p.h = (int32_t)rows[l];
                p.w = (int32_t)cols[l];
                p.trans = rows[l] > cols[l] ? 1 : 0;
                probs.push_back(p);
            } else {
                const int64_t R = ceil_div(rows[l], Th), C = ceil_div(cols[l], Tw);
                p.trans = Th > Tw ? 1 : 0;  // the orientation rule on a tall tile
                for (int64_t r = 0; r < R; ++r)
                    for (int64_t q = 0; q < C; ++q) {
                        p.row0 = r * Th;
                        p.col0 = q * Tw;
                        p.h = (int32_t)std::min<int64_t>(Th, rows[l] - r * Th);
                        p.w = (int32_t)std::min<int64_t>(Tw, cols[l] - q * Tw);
                        probs.push_back(p);
                    }
            }
        }
    }

    hipStream_t hs = static_cast<hipStream_t>(stream);
    int cur = 0, dev = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return himuon::set_hip_error(e);
    dev = cur;
    if (hs) {
        e = hipStreamGetDevice(hs, &dev);
        if (e != hipSuccess) return himuon::set_hip_error(e);
    }
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return himuon::set_hip_error(e);

    // every GEMM plan exists before anything is enqueued
    std::lock_guard<std::mutex> enqueue_lock(g_enqueue_mu);
    hipblasLtHandle_t lt = nullptr;
    int status = HIMUON_OK;
    for (const Group& g : groups) {
        const int64_t small = g.count / g.n_chunks, big = ceil_div(g.count, g.n_chunks);
        Plan* pl = nullptr;
        status = get_plan(dev, g.m, g.n, (int)big, op, &lt, &pl);
        if (status == HIMUON_OK && small != big && small > 0) status = get_plan(dev, g.m, g.n, (int)small, op, &lt, &pl);
        if (status != HIMUON_OK) break;
    }

    // workspace: table | partials | X0 | X1 | A | B | hipBLASLt scratch
    uint8_t* const ws = static_cast<uint8_t*>(workspace);
    GemmProb* const table = reinterpret_cast<GemmProb*>(ws);
    size_t off = align_up((size_t)total * sizeof(GemmProb));
    size_t part_max = 0, buf_max = 0;
    const size_t es = op_size(op);
    for (const Group& g : groups) {
        part_max = std::max(part_max, (size_t)g.cap * g.nparts * sizeof(double));
        buf_max = std::max(buf_max, 2 * align_up((size_t)g.cap * g.m * g.n * es) + 2 * align_up((size_t)g.cap * g.m * g.m * es));
    }
    double* const partial = reinterpret_cast<double*>(ws + off);
    off += align_up(part_max);
    uint8_t* const bufs = ws + off;
    void* const lt_ws = ws + off + buf_max;

    if (status == HIMUON_OK) status = himuon::upload_table(probs.data(), probs.size() * sizeof(GemmProb), table, hs, dev);
    for (const Group& g : groups) {
        if (status != HIMUON_OK) break;
        const size_t xb = align_up((size_t)g.cap * g.m * g.n * es), ab = align_up((size_t)g.cap * g.m * g.m * es);
        void* X[2] = {bufs, bufs + xb};
        void* A = bufs + 2 * xb;
        void* B = bufs + 2 * xb + ab;
        const double s = iterate_scale(op, g.m);
        const float alpha2 = (float)((double)c / (s * s * s * s)), beta2 = (float)((double)b / (s * s));
        for (int64_t ci = 0; ci < g.n_chunks && status == HIMUON_OK; ++ci) {
            const int64_t p0 = (int64_t)(((__int128)ci * g.count) / g.n_chunks);
            const int64_t p1 = (int64_t)(((__int128)(ci + 1) * g.count) / g.n_chunks);
            const int np = (int)(p1 - p0);
            const GemmProb* tp = table + g.first + p0;
            Plan* pl = nullptr;
            status = get_plan(dev, g.m, g.n, np, op, &lt, &pl);
            if (status != HIMUON_OK) break;
            if ((e = himuon::launch_gemm_norm_partials(sto, tp, np, g.nparts, partial, opt, hs)) != hipSuccess ||
                (e = himuon::launch_gemm_gather(sto, op, tp, np, g.m, g.n, g.nparts, partial, s, X[0], opt, hs)) !=
                    hipSuccess) {
                status = himuon::set_hip_error(e);
                break;
            }
            int cur_x = 0;
            for (int k = 0; k < K && status == HIMUON_OK; ++k) {
                void* x = X[cur_x];
                void* xn = X[cur_x ^ 1];
                status = run_gemm(lt, pl->gram, 1.f, x, x, 0.f, A, A, lt_ws, hs);
                if (status == HIMUON_OK) status = run_gemm(lt, pl->poly, alpha2, A, A, beta2, A, B, lt_ws, hs);
                if (status == HIMUON_OK) status = run_gemm(lt, pl->apply, 1.f, x, B, a, x, xn, lt_ws, hs);
                cur_x ^= 1;
            }
            if (status == HIMUON_OK &&
                (e = himuon::launch_gemm_scatter(sto, op, tp, np, g.m, g.n, (float)(1.0 / s), X[cur_x], opt, hs)) !=
                    hipSuccess)
                status = himuon::set_hip_error(e);
        }
    }
    if (dev != cur) (void)hipSetDevice(cur);
    return status;
}

size_t gemm_path_workspace(int64_t n_mats, const int64_t* rows, const int64_t* cols, int Th, int Tw, int dtype, int compute,
                           int K, float a, float b, float c, size_t chunk_budget_bytes)
{
    std::vector<Group> groups;
    if (plan_groups(n_mats, rows, cols, Th, Tw, groups, nullptr) != HIMUON_OK) return 0;
    int m_max = 0;
    for (const Group& g : groups) m_max = std::max(m_max, g.m);
    GemmOperand op;
    if (dtype != HIMUON_F32 && dtype != HIMUON_BF16) return 0;
    if (resolve_operand(dtype, compute, K, a, b, c, m_max, &op) != HIMUON_OK) return 0;
    size_t ws = 0;
    if (plan_chunks(groups, op, chunk_budget_bytes, &ws) != HIMUON_OK) return 0;
    return ws;
}

}  // namespace himuon

extern "C" {

size_t himuon_ns_gemm_hw_workspace_size(int64_t n_mats, const int64_t* rows, const int64_t* cols, int Th, int Tw,
                                        int dtype, int compute, int K, float a, float b, float c,
                                        size_t chunk_budget_bytes)
{
    return himuon::gemm_path_workspace(n_mats, rows, cols, Th, Tw, dtype, compute, K, a, b, c, chunk_budget_bytes);
}

size_t himuon_ns_gemm_workspace_size(int64_t n_mats, const int64_t* rows, const int64_t* cols, int T, int dtype,
                                     int compute, int K, float a, float b, float c, size_t chunk_budget_bytes)
{
    if (T < 0) return 0;
    return himuon::gemm_path_workspace(n_mats, rows, cols, T, T, dtype, compute, K, a, b, c, chunk_budget_bytes);
}

int himuon_ns_gemm_hw(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, const int64_t* rows,
                      const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int Th, int Tw, int K, float a,
                      float b, float c, int dtype, int compute, void* workspace, size_t workspace_bytes,
                      size_t chunk_budget_bytes, void* stream)
{
    return himuon::run_gemm_path(n_mats, in_ptrs, out_ptrs, nullptr, nullptr, rows, cols, ld_in, ld_out, Th, Tw, K, a,
                                 b, c, dtype, compute, workspace, workspace_bytes, chunk_budget_bytes, stream, nullptr);
}

int himuon_ns_gemm(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs, const int64_t* rows,
                   const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int T, int K, float a, float b,
                   float c, int dtype, int compute, void* workspace, size_t workspace_bytes,
                   size_t chunk_budget_bytes, void* stream)
{
    if (T < 0) return HIMUON_ERR_INVALID_ARG;
    return himuon::run_gemm_path(n_mats, in_ptrs, out_ptrs, nullptr, nullptr, rows, cols, ld_in, ld_out, T, T, K, a, b,
                                 c, dtype, compute, workspace, workspace_bytes, chunk_budget_bytes, stream, nullptr);
}


int himuon_gemm_tune_hw(int64_t n_mats, const int64_t* rows, const int64_t* cols, int Th, int Tw, int dtype,
                        int compute, int K, float a, float b, float c, void* workspace, size_t workspace_bytes,
                        size_t chunk_budget_bytes, void* stream)
{
    if (n_mats < 1 || !rows || !cols || K < 0 || !valid_tiling(Th, Tw) || !isfinite(a) || !isfinite(b) ||
        !isfinite(c))
        return HIMUON_ERR_INVALID_ARG;
    if (dtype != HIMUON_F32 && dtype != HIMUON_BF16) return HIMUON_ERR_INVALID_ARG;
    if (compute < HIMUON_COMPUTE_DEFAULT || compute > HIMUON_COMPUTE_BF16) return HIMUON_ERR_INVALID_ARG;
    std::vector<Group> groups;
    int st = plan_groups(n_mats, rows, cols, Th, Tw, groups, nullptr);
    if (st != HIMUON_OK) return st;
    int m_max = 0;
    int64_t total = 0;
    for (const Group& g : groups) {
        m_max = std::max(m_max, g.m);
        total += g.count;
    }
    GemmOperand op;
    st = resolve_operand(dtype, compute, K, a, b, c, m_max, &op);
    if (st != HIMUON_OK) return st;
    size_t need = 0;
    st = plan_chunks(groups, op, chunk_budget_bytes, &need);
    if (st != HIMUON_OK) return st;
    if (!workspace || workspace_bytes < need) return HIMUON_ERR_WORKSPACE;

    hipStream_t hs = static_cast<hipStream_t>(stream);
    int cur = 0, dev = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return himuon::set_hip_error(e);
    dev = cur;
    if (hs) {
        e = hipStreamGetDevice(hs, &dev);
        if (e != hipSuccess) return himuon::set_hip_error(e);
    }
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return himuon::set_hip_error(e);
    std::lock_guard<std::mutex> enqueue_lock(g_enqueue_mu);
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if ((e = hipEventCreate(&e0)) != hipSuccess || (e = hipEventCreate(&e1)) != hipSuccess) {
        if (e0) (void)hipEventDestroy(e0);
        if (dev != cur) (void)hipSetDevice(cur);
        return himuon::set_hip_error(e);
    }
    const size_t es = op_size(op);
    size_t part_max = 0, buf_max = 0;
    for (const Group& g : groups) {
        part_max = std::max(part_max, (size_t)g.cap * g.nparts * sizeof(double));
        buf_max = std::max(buf_max, 2 * align_up((size_t)g.cap * g.m * g.n * es) + 2 * align_up((size_t)g.cap * g.m * g.m * es));
    }
    uint8_t* const bufs = static_cast<uint8_t*>(workspace) + align_up((size_t)total * sizeof(GemmProb)) + align_up(part_max);
    void* const lt_ws = bufs + buf_max;
    for (const Group& g : groups) {
        if (st != HIMUON_OK) break;
        const size_t xb = align_up((size_t)g.cap * g.m * g.n * es), ab = align_up((size_t)g.cap * g.m * g.m * es);
        uint8_t* const X0 = bufs;
        uint8_t* const X1 = bufs + xb;
        uint8_t* const A = bufs + 2 * xb;
        uint8_t* const B = bufs + 2 * xb + ab;
        const double s = iterate_scale(op, g.m);
        const float alpha2 = (float)((double)c / (s * s * s * s)), beta2 = (float)((double)b / (s * s));
        const int64_t sizes[2] = {ceil_div(g.count, g.n_chunks), g.count / g.n_chunks};
        for (int k = 0; k < 2 && st == HIMUON_OK; ++k) {
            if (sizes[k] < 1 || (k == 1 && sizes[1] == sizes[0])) continue;
            hipblasLtHandle_t lt = nullptr;
            Plan* pl = nullptr;
            st = get_plan(dev, g.m, g.n, (int)sizes[k], op, &lt, &pl);
            if (st != HIMUON_OK || pl->tuned) continue;
            st = tune_gemm(lt, pl->gram, 1.f, X0, X0, 0.f, A, A, lt_ws, hs, e0, e1);
            if (st == HIMUON_OK) st = tune_gemm(lt, pl->poly, alpha2, A, A, beta2, A, B, lt_ws, hs, e0, e1);
            if (st == HIMUON_OK) st = tune_gemm(lt, pl->apply, 1.f, X0, B, a, X0, X1, lt_ws, hs, e0, e1);
            if (st == HIMUON_OK) pl->tuned = true;
        }
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (dev != cur) (void)hipSetDevice(cur);
    return st;
}

int himuon_gemm_tune(int64_t n_mats, const int64_t* rows, const int64_t* cols, int T, int dtype, int compute, int K,
                     float a, float b, float c, void* workspace, size_t workspace_bytes, size_t chunk_budget_bytes,
                     void* stream)
{
    if (T < 0) return HIMUON_ERR_INVALID_ARG;
    return himuon_gemm_tune_hw(n_mats, rows, cols, T, T, dtype, compute, K, a, b, c, workspace, workspace_bytes,
                               chunk_budget_bytes, stream);
}

}  // extern "C"
