// The HiMuon optimizer step (Alg. 1) over a batch of parameter matrices:
//   M <- beta M + G;  Ghat = G + beta M (Nesterov) or M;
//   U = Phi_K(Ghat) when T = 0 (the branch T = infinity) or T >= max(H, W),
//       else Phi_{K,T}(Ghat);
//   W <- (1 - lr lambda) W - lr tau U, tau = c sqrt(max(H, W)) on the full
//       branch and c sqrt(T) when tiled (Sec. 4.2, eq. scaled_update).
// Three execution routes, chosen from T and the types:
//   - T in {32, 64, 128} (fp32 storage; bf16 storage with bf16 operands; bf16
//     storage with fp16 operands when c > 0): the step inside the fused tile
//     kernel (its gather forms the momentum and the lookahead, its
//     write-back the weight update), so every matrix is read and written once;
//   - T = 256, or c <= 0 with fp16 operands: an element-wise prologue
//     (momentum and lookahead into a contiguous buffer), the tiled map in
//     place on that buffer, and an element-wise epilogue (decay and update);
//     matrices are taken in consecutive groups whose buffers fit the chunk
//     budget;
//   - otherwise (T = 0, large tiles such as 512): the library-GEMM path with
//     the momentum fused into its norm and gather kernels and the update into
//     its scatter kernel.
#include "himuon_internal.h"
#include "ns_gemm_path.h"
#include "optim_kernels.h"
#include "../../include/himuon.h"

#include <algorithm>
#include <math.h>
#include <vector>

namespace {

using himuon::GemmStore;
using himuon::OptArgs;
using himuon::StepDesc;

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool fused_route(int T, int dtype, int compute, int K, float a, float b, float c)
{
    if (T != 32 && T != 64 && T != 128 && T != 256) return false;
    const int op = himuon_select_compute(dtype, compute, K, a, b, c);
    if (op < 0) return false;
    const himuon::Storage st = dtype == HIMUON_BF16 ? himuon::Storage::BF16 : himuon::Storage::F32;
    return himuon::has_kernel(T, st, (himuon::Operand)op);
}

// The step can run inside the tile kernel (see the file comment).
bool in_kernel_route(int T, int dtype, int compute, int K, float a, float b, float c)
{
    if (!fused_route(T, dtype, compute, K, a, b, c)) return false;
    const int op = himuon_select_compute(dtype, compute, K, a, b, c);
    const himuon::Storage st = dtype == HIMUON_BF16 ? himuon::Storage::BF16 : himuon::Storage::F32;
    return himuon::has_step_kernel(T, st, (himuon::Operand)op, c);
}

size_t elem_size(int dtype) { return dtype == HIMUON_BF16 ? 2 : 4; }

// Consecutive matrix groups [bounds[i], bounds[i+1]) whose contiguous
// buffers fit `budget` (0: one group); the largest group's buffer bytes.
int plan_step_groups(int64_t n_mats, const int64_t* rows, const int64_t* cols, int dtype, size_t budget,
                     std::vector<int64_t>* bounds, size_t* buf_max)
{
    const size_t es = elem_size(dtype);
    bounds->assign(1, 0);
    size_t cur = 0, mx = 0;
    for (int64_t l = 0; l < n_mats; ++l) {
        const size_t bytes = align_up((size_t)rows[l] * (size_t)cols[l] * es);
        if (budget && bytes > budget) return HIMUON_ERR_WORKSPACE;
        if (budget && cur + bytes > budget) {
            bounds->push_back(l);
            cur = 0;
        }
        cur += bytes;
        mx = std::max(mx, cur);
    }
    bounds->push_back(n_mats);
    *buf_max = mx;
    return HIMUON_OK;
}

size_t fused_route_workspace(int64_t n_mats, size_t buf_max)
{
    return align_up(buf_max) + align_up((size_t)n_mats * sizeof(StepDesc)) + himuon_ns_tiled_workspace_size(n_mats);
}

float tau_of(int64_t rows, int64_t cols, int T, float scale_c)
{
    const int64_t big = std::max(rows, cols);
    const bool full = T == 0 || T >= big;
    return (float)((double)scale_c * sqrt((double)(full ? big : T)));
}

}  // namespace

extern "C" {

size_t himuon_step_workspace_size(int64_t n_mats, const int64_t* rows, const int64_t* cols, int T, int dtype,
                                  int compute, int K, float a, float b, float c, size_t chunk_budget_bytes)
{
    if (n_mats < 1 || !rows || !cols || T < 0 || K < 0) return 0;
    if (dtype != HIMUON_F32 && dtype != HIMUON_BF16) return 0;
    for (int64_t l = 0; l < n_mats; ++l)
        if (rows[l] < 1 || cols[l] < 1) return 0;
    if (in_kernel_route(T, dtype, compute, K, a, b, c)) return himuon::tiled_workspace(n_mats, true);
    if (fused_route(T, dtype, compute, K, a, b, c)) {
        std::vector<int64_t> bounds;
        size_t buf_max = 0;
        if (plan_step_groups(n_mats, rows, cols, dtype, chunk_budget_bytes, &bounds, &buf_max) != HIMUON_OK) return 0;
        return fused_route_workspace(n_mats, buf_max);
    }
    return himuon::gemm_path_workspace(n_mats, rows, cols, T, T, dtype, compute, K, a, b, c, chunk_budget_bytes);
}

int himuon_step(int64_t n_mats, void* const* weights, const void* const* grads, void* const* moms,
                const int64_t* rows, const int64_t* cols, const int64_t* ld, int T, int K, float a, float b, float c,
                float lr, float momentum, float weight_decay, int nesterov, float scale_c, int dtype, int compute,
                void* workspace, size_t workspace_bytes, size_t chunk_budget_bytes, void* stream)
{
    // ---- validation: nothing is enqueued unless every check passes
    if (n_mats < 1 || n_mats > INT32_MAX || !weights || !grads || !moms || !rows || !cols) return HIMUON_ERR_INVALID_ARG;
    if (K < 0 || T < 0 || !isfinite(a) || !isfinite(b) || !isfinite(c)) return HIMUON_ERR_INVALID_ARG;
    if (!isfinite(lr) || !isfinite(momentum) || !isfinite(weight_decay) || !isfinite(scale_c))
        return HIMUON_ERR_INVALID_ARG;
    if (dtype != HIMUON_F32 && dtype != HIMUON_BF16) return HIMUON_ERR_INVALID_ARG;
    if (compute < HIMUON_COMPUTE_DEFAULT || compute > HIMUON_COMPUTE_BF16) return HIMUON_ERR_INVALID_ARG;
    std::vector<float> tau((size_t)n_mats);
    const int64_t mult = dtype == HIMUON_BF16 ? 8 : 4;
    for (int64_t l = 0; l < n_mats; ++l) {
        if (!weights[l] || !grads[l] || !moms[l] || rows[l] < 1 || cols[l] < 1) return HIMUON_ERR_INVALID_ARG;
        if (weights[l] == grads[l] || weights[l] == moms[l] || grads[l] == moms[l]) return HIMUON_ERR_INVALID_ARG;
        const int64_t li = ld ? ld[l] : cols[l];
        if (li < cols[l] || rows[l] > INT64_MAX / li) return HIMUON_ERR_INVALID_ARG;
        if (rows[l] > INT32_MAX || cols[l] > INT32_MAX) return HIMUON_ERR_UNSUPPORTED;
        tau[(size_t)l] = tau_of(rows[l], cols[l], T, scale_c);
        if (!isfinite(tau[(size_t)l])) return HIMUON_ERR_INVALID_ARG;
    }
    OptArgs opt;
    opt.beta = momentum;
    opt.decay = (float)(1.0 - (double)lr * (double)weight_decay);
    opt.lr = lr;
    opt.nesterov = nesterov ? 1 : 0;

    if (!fused_route(T, dtype, compute, K, a, b, c)) {
        std::vector<const void*> in((size_t)n_mats);
        std::vector<int64_t> lds((size_t)n_mats);
        for (int64_t l = 0; l < n_mats; ++l) {
            in[(size_t)l] = grads[l];
            lds[(size_t)l] = ld ? ld[l] : cols[l];
        }
        return himuon::run_gemm_path(n_mats, in.data(), weights, moms, tau.data(), rows, cols, lds.data(), lds.data(),
                                     T, T, K, a, b, c, dtype, compute, workspace, workspace_bytes, chunk_budget_bytes,
                                     stream, &opt);
    }

    if (in_kernel_route(T, dtype, compute, K, a, b, c)) {
        std::vector<himuon::OptDesc> od((size_t)n_mats);
        std::vector<const void*> in((size_t)n_mats);
        for (int64_t l = 0; l < n_mats; ++l) {
            od[(size_t)l].mom = moms[l];
            od[(size_t)l].tau = tau[(size_t)l];
            od[(size_t)l].pad_ = 0;
            in[(size_t)l] = grads[l];
        }
        return himuon::run_tiled(n_mats, in.data(), weights, rows, cols, ld, ld, T, K, a, b, c, dtype, compute,
                                 workspace, workspace_bytes, chunk_budget_bytes, stream, od.data(), opt.beta,
                                 opt.decay, opt.lr, opt.nesterov);
    }

    // ---- fused-kernel route with element-wise prologue and epilogue
    std::vector<int64_t> bounds;
    size_t buf_max = 0;
    int st = plan_step_groups(n_mats, rows, cols, dtype, chunk_budget_bytes, &bounds, &buf_max);
    if (st != HIMUON_OK) return st;
    if (!workspace || workspace_bytes < fused_route_workspace(n_mats, buf_max)) return HIMUON_ERR_WORKSPACE;
    uint8_t* const ws = static_cast<uint8_t*>(workspace);
    uint8_t* const buf = ws;
    StepDesc* const dtab = reinterpret_cast<StepDesc*>(ws + align_up(buf_max));
    void* const ns_ws = ws + align_up(buf_max) + align_up((size_t)n_mats * sizeof(StepDesc));
    const size_t ns_ws_bytes = himuon_ns_tiled_workspace_size(n_mats);
    const size_t es = elem_size(dtype);

    std::vector<StepDesc> descs((size_t)n_mats);
    std::vector<void*> bufs((size_t)n_mats);
    std::vector<int64_t> group_chunks(bounds.size() - 1, 0);
    for (size_t gi = 0; gi + 1 < bounds.size(); ++gi) {
        size_t off = 0;
        for (int64_t l = bounds[gi]; l < bounds[gi + 1]; ++l) {
            StepDesc& d = descs[(size_t)l];
            d.w = weights[l];
            d.g = grads[l];
            d.m = moms[l];
            d.buf = buf + off;
            bufs[(size_t)l] = d.buf;
            off += align_up((size_t)rows[l] * (size_t)cols[l] * es);
            d.rows = rows[l];
            d.cols = cols[l];
            d.ld = ld ? ld[l] : cols[l];
            d.tau = tau[(size_t)l];
            d.vec = ((uintptr_t)d.w % 16 == 0 && (uintptr_t)d.g % 16 == 0 && (uintptr_t)d.m % 16 == 0 &&
                     d.ld % mult == 0) ? 1 : 0;
            d.vec_buf = d.cols % mult == 0 ? 1 : 0;
            group_chunks[gi] = std::max<int64_t>(group_chunks[gi], d.rows * ((d.cols + 7) / 8));
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
    const GemmStore sto = dtype == HIMUON_BF16 ? GemmStore::BF16 : GemmStore::F32;
    int status = himuon::upload_table(descs.data(), descs.size() * sizeof(StepDesc), dtab, hs, dev);
    for (size_t gi = 0; gi + 1 < bounds.size() && status == HIMUON_OK; ++gi) {
        const int64_t l0 = bounds[gi], nl = bounds[gi + 1] - bounds[gi];
        if ((e = himuon::launch_step_lookahead(sto, dtab + l0, (int)nl, group_chunks[gi], opt, hs)) != hipSuccess) {
            status = himuon::set_hip_error(e);
            break;
        }
        status = himuon_ns_tiled(nl, const_cast<const void* const*>(bufs.data() + l0), bufs.data() + l0, rows + l0,
                                 cols + l0, nullptr, nullptr, T, K, a, b, c, dtype, compute, ns_ws, ns_ws_bytes, 0,
                                 hs);
        if (status != HIMUON_OK) break;
        if ((e = himuon::launch_step_apply(sto, dtab + l0, (int)nl, group_chunks[gi], opt, hs)) != hipSuccess)
            status = himuon::set_hip_error(e);
    }
    if (dev != cur) (void)hipSetDevice(cur);
    return status;
}

}  // extern "C"
