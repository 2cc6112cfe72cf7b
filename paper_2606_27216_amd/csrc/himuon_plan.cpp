// Plans: a himuon_ns_tiled, himuon_ns_gemm or himuon_step call recorded once
// into a HIP graph, replayed by himuon_plan_launch with no host work but one
// graph launch. This is the graph-captured cross-layer step of the optimizer-step
// study (Sec. 6.4) and the graph-capture state that the runtime tile-size
// reconfiguration rebuilds when T changes (Sec. 4.4.3).
//
// Recording runs the ordinary entry point on a private stream under stream
// capture (relaxed mode). Its descriptor tables are copied from pinned
// buffers that the plan owns (upload_table's recording mode), so every
// replay copies the same tables into the caller's workspace before the
// kernels that read them; the graph holds kernel and copy nodes only.
#include "himuon_internal.h"
#include "../../include/himuon.h"

struct himuon_plan {
    int dev = -1;
    hipStream_t stream = nullptr;  // the recording stream
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    himuon::PlanRecording rec;
};

namespace {

void release(himuon_plan* p)
{
    if (!p) return;
    int cur = 0;
    const bool switched = hipGetDevice(&cur) == hipSuccess && p->dev >= 0 && cur != p->dev &&
                          hipSetDevice(p->dev) == hipSuccess;
    if (p->exec) (void)hipGraphExecDestroy(p->exec);
    if (p->graph) (void)hipGraphDestroy(p->graph);
    if (p->stream) (void)hipStreamDestroy(p->stream);
    for (void* h : p->rec.host_buffers) (void)hipHostFree(h);
    if (switched) (void)hipSetDevice(cur);
    delete p;
}

// Records `call(stream)` into a new plan on the current device.
template <class Call> int record(himuon_plan** out, Call call)
{
    if (!out) return HIMUON_ERR_INVALID_ARG;
    *out = nullptr;
    himuon_plan* p = new himuon_plan();
    hipError_t e = hipGetDevice(&p->dev);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&p->stream, hipStreamNonBlocking);
    if (e != hipSuccess) {
        release(p);
        return himuon::set_hip_error(e);
    }
    int st = himuon::gemm_handle_ready(p->dev);  // not inside the capture
    if (st == HIMUON_OK) {
        e = hipStreamBeginCapture(p->stream, hipStreamCaptureModeRelaxed);
        if (e != hipSuccess) st = himuon::set_hip_error(e);
    }
    if (st == HIMUON_OK) {
        himuon::g_recording = &p->rec;
        st = call(p->stream);
        himuon::g_recording = nullptr;
        e = hipStreamEndCapture(p->stream, &p->graph);
        if (st == HIMUON_OK && e != hipSuccess) st = himuon::set_hip_error(e);
    }
    if (st == HIMUON_OK) {
        e = hipGraphInstantiate(&p->exec, p->graph, nullptr, nullptr, 0);
        if (e != hipSuccess) st = himuon::set_hip_error(e);
    }
    if (st != HIMUON_OK) {
        release(p);
        return st;
    }
    *out = p;
    return HIMUON_OK;
}

}  // namespace

extern "C" {

int himuon_plan_ns_tiled(himuon_plan_t** plan, int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs,
                         const int64_t* rows, const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int T,
                         int K, float a, float b, float c, int dtype, int compute, void* workspace,
                         size_t workspace_bytes, size_t chunk_budget_bytes)
{
    return record(plan, [&](hipStream_t s) {
        return himuon_ns_tiled(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, T, K, a, b, c, dtype, compute,
                               workspace, workspace_bytes, chunk_budget_bytes, s);
    });
}

int himuon_plan_ns_gemm(himuon_plan_t** plan, int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs,
                        const int64_t* rows, const int64_t* cols, const int64_t* ld_in, const int64_t* ld_out, int T,
                        int K, float a, float b, float c, int dtype, int compute, void* workspace,
                        size_t workspace_bytes, size_t chunk_budget_bytes)
{
    return record(plan, [&](hipStream_t s) {
        return himuon_ns_gemm(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, T, K, a, b, c, dtype, compute,
                              workspace, workspace_bytes, chunk_budget_bytes, s);
    });
}

int himuon_plan_step(himuon_plan_t** plan, int64_t n_mats, void* const* weights, const void* const* grads,
                     void* const* moms, const int64_t* rows, const int64_t* cols, const int64_t* ld, int T, int K,
                     float a, float b, float c, float lr, float momentum, float weight_decay, int nesterov,
                     float scale_c, int dtype, int compute, void* workspace, size_t workspace_bytes,
                     size_t chunk_budget_bytes)
{
    return record(plan, [&](hipStream_t s) {
        return himuon_step(n_mats, weights, grads, moms, rows, cols, ld, T, K, a, b, c, lr, momentum, weight_decay,
                           nesterov, scale_c, dtype, compute, workspace, workspace_bytes, chunk_budget_bytes, s);
    });
}

int himuon_plan_launch(const himuon_plan_t* plan, void* stream)
{
    if (!plan || !plan->exec) return HIMUON_ERR_INVALID_ARG;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    int cur = 0, dev = 0;
    int st = himuon::stream_device(hs, &cur, &dev);
    if (st != HIMUON_OK) return st;
    if (dev != plan->dev) st = HIMUON_ERR_INVALID_ARG;
    if (st == HIMUON_OK) {
        const hipError_t e = hipGraphLaunch(plan->exec, hs);
        if (e != hipSuccess) st = himuon::set_hip_error(e);
    }
    if (dev != cur) (void)hipSetDevice(cur);
    return st;
}

void himuon_plan_destroy(himuon_plan_t* plan) { release(plan); }

}  // extern "C"
