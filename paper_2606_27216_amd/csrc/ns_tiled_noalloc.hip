// himuon_ns_tiled_noalloc: the fused tiled map for callers that cannot
// allocate (code under stream capture, tight serving loops). It runs the same
// kernels as himuon_ns_tiled; the only device memory the kernels need beyond
// the caller's matrices, the per-matrix descriptor table, lives in a
// file-scope device array instead of a caller workspace, and reaches it
// through the arguments of small upload kernels instead of a host staging
// copy. Nothing here calls an allocating routine, host or device.
#include "himuon_internal.h"
#include "../../include/himuon.h"

#include <mutex>
#include <string.h>

namespace {

using himuon::MatDesc;

constexpr int kMaxMats = HIMUON_NOALLOC_MAX_MATS;
constexpr int kPerUpload = 48;                // descriptors one upload launch carries (3 KiB of arguments)
constexpr int kWordsPerDesc = (int)(sizeof(MatDesc) / 16);
constexpr int kMaxDevices = 64;
static_assert(sizeof(MatDesc) % 16 == 0, "descriptor is a whole number of 16-byte words");

// The descriptor table of the last call on this device (64 KiB). Every call
// on a device writes its own entries [0, n_mats) before its tile kernels read
// them, so nothing needs clearing; calls that overlap on one device race.
static __device__ __align__(256) MatDesc scratch[kMaxMats];

struct DescWords {
    uint4 w[kPerUpload * kWordsPerDesc];
};

// One thread per 16-byte word: table[i] = words.w[i] for i < n_words.
__global__ void __launch_bounds__(kPerUpload * kWordsPerDesc) upload_descs(const DescWords words, int n_words,
                                                                            uint4* table)
{
    const int i = threadIdx.x;
    if (i < n_words) table[i] = words.w[i];
}

std::mutex g_mu;
void* g_table[kMaxDevices];  // device address of `scratch` on each device; null until looked up

// `scratch`'s address on device `dev`, which must be current: the array's
// host-side name is only a stand-in, each device holds its own copy.
int table_address(int dev, void** ptr)
{
    if (dev < 0 || dev >= kMaxDevices) return himuon::set_hip_error(hipErrorInvalidDevice);
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_table[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return himuon::set_hip_error(e);
        if (!p) return himuon::set_hip_error(hipErrorInvalidSymbol);
        g_table[dev] = p;
    }
    *ptr = g_table[dev];
    return HIMUON_OK;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

extern "C" int himuon_ns_tiled_noalloc(int64_t n_mats, const void* const* in_ptrs, void* const* out_ptrs,
                                       const int64_t* rows, const int64_t* cols, const int64_t* ld_in,
                                       const int64_t* ld_out, int T, int K, float a, float b, float c, int dtype,
                                       int compute, size_t chunk_budget_bytes, void* stream)
{
    // ---- validation: nothing is enqueued unless every check passes
    int op = 0;
    const bool t_ok = T == 32 || T == 64 || T == 128 || T == 256;
    int s = himuon::validate_tiled(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, t_ok ? T : 32, K, a, b, c,
                                   dtype, compute, &op);
    if (s != HIMUON_OK) return s;
    if (!t_ok) return HIMUON_ERR_UNSUPPORTED;
    const himuon::Storage st = dtype == HIMUON_BF16 ? himuon::Storage::BF16 : himuon::Storage::F32;
    const himuon::Operand opnd = (himuon::Operand)op;
    // (the GEMM route of 256-tiles without a fused kernel needs a workspace)
    if (!himuon::has_kernel(T, st, opnd)) return HIMUON_ERR_UNSUPPORTED;
    if (n_mats > kMaxMats) return HIMUON_ERR_WORKSPACE;
    int64_t total = 0, n_chunks = 0;
    s = himuon::plan_tiled_chunks(n_mats, rows, cols, T, T, dtype, chunk_budget_bytes, &total, &n_chunks);
    if (s != HIMUON_OK) return s;

    hipStream_t hs = static_cast<hipStream_t>(stream);
    int cur = 0, dev = 0;
    s = himuon::stream_device(hs, &cur, &dev);
    if (s != HIMUON_OK) return s;
    void* table = nullptr;
    int status = table_address(dev, &table);

    // ---- descriptor table: carried by the tile kernels' own arguments for a
    // call of at most himuon::kInlineMats matrices, else written to `scratch`
    // in batches carried by the arguments of upload kernels
    const bool inl = n_mats <= himuon::kInlineMats;
    MatDesc inline_descs[himuon::kInlineMats];
    DescWords words;
    int64_t next = 0;
    if (inl) {
        for (int64_t m = 0; m < n_mats; ++m) {
            inline_descs[m] = himuon::make_desc(in_ptrs[m], out_ptrs[m], rows[m], cols[m],
                                                ld_in ? ld_in[m] : cols[m], ld_out ? ld_out[m] : cols[m], next, T,
                                                dtype, nullptr);
            next += ceil_div(rows[m], T) * ceil_div(cols[m], T);
        }
    }
    for (int64_t m0 = 0; !inl && m0 < n_mats && status == HIMUON_OK; m0 += kPerUpload) {
        const int n = (int)(n_mats - m0 < kPerUpload ? n_mats - m0 : kPerUpload);
        memset(&words, 0, sizeof(words));
        for (int j = 0; j < n; ++j) {
            const int64_t m = m0 + j;
            const MatDesc d = himuon::make_desc(in_ptrs[m], out_ptrs[m], rows[m], cols[m],
                                                ld_in ? ld_in[m] : cols[m], ld_out ? ld_out[m] : cols[m], next, T,
                                                dtype, nullptr);
            memcpy(&words.w[j * kWordsPerDesc], &d, sizeof(MatDesc));
            next += ceil_div(rows[m], T) * ceil_div(cols[m], T);
        }
        hipLaunchKernelGGL(upload_descs, dim3(1), dim3(kPerUpload * kWordsPerDesc), 0, hs, words,
                           n * kWordsPerDesc, static_cast<uint4*>(table) + m0 * kWordsPerDesc);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) status = himuon::set_hip_error(e);
    }
    if (status == HIMUON_OK) {
        himuon::KernelArgs ka = himuon::make_kernel_args(static_cast<const MatDesc*>(table), n_mats, K, a, b, c);
        if (inl) himuon::set_inline_tables(ka, inline_descs, nullptr, n_mats);
        status = himuon::launch_chunks(T, st, opnd, ka, total, n_chunks, hs);
    }
    if (dev != cur) (void)hipSetDevice(cur);
    return status;
}
