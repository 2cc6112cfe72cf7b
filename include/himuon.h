/*
 * himuon.h — C ABI of the MI355X (gfx950) tiled Newton–Schulz library.
 *
 * The library evaluates the tiled Newton–Schulz map of Hierarchical Muon,
 *
 *     Phi_{K,T}(G) = B_T^{-1}( { Phi_K(G_rc) }_{r,c} )        eq. (tiled_ns), Sec. 4.1
 *
 * on a batch of matrices in one call:
 *   - B_T (Sec. 2.1, eq. tiling_operator) pads an H x W matrix with zeros to
 *     (RT) x (CT), R = ceil(H/T), C = ceil(W/T), and cuts it into T x T tiles;
 *     B_T^{-1} reassembles them and drops the padding;
 *   - Phi_K (Sec. 2.2, eqs. ns_iteration, ns_quintic, phi_k_def) normalises
 *     a tile, X_0 = S/||S||_F (Phi_K(0) = 0), and applies K steps of
 *     X <- (aI + bA + cA^2) X with A = X X^T;
 *   - tiles of every matrix in the call are batched into shared launches
 *     ("cross-layer batching", Sec. 4.4.2) and split into the fewest balanced
 *     chunks that fit a memory budget (memory-bounded chunking, Sec. 4.4.2).
 *
 * All entry points are plain C: host pointers for the small per-matrix
 * arrays, device pointers for matrix data and workspace, and a HIP stream
 * passed as void* (a hipStream_t; NULL is the null stream). No entry point
 * allocates device memory or synchronises the device on the compute path.
 * A fused-kernel call over at most 32 matrices carries its descriptor table
 * in the kernels' own launch arguments. Other calls copy their descriptor
 * tables to the workspace from a ring of pinned host slots (allocated on
 * first use, reused once the copy that last used a slot has completed), so
 * calls are not meant for stream capture into a HIP graph: a captured copy
 * would read whatever a slot holds at replay (plans, below, record such
 * calls safely).
 *
 * Matrices are row-major: element (i, j) of matrix l sits at
 * ptr_l + i*ld_l + j (in elements). One call uses one storage dtype for all
 * inputs and outputs.
 *
 * Threads: every entry point may be called from several host threads at
 * once, each on its own stream (or the same one). The library's shared host
 * state (staging ring, per-device GEMM handle and plans, cached bounds) is
 * locked, the last HIP error is per thread, and calls that run library GEMMs
 * (himuon_ns_gemm*, himuon_gemm_tune*, the GEMM route of himuon_ns_tiled and
 * himuon_step) enqueue one thread at a time; the device work of calls on
 * different streams still overlaps. Calls whose output buffers overlap race
 * on the device as any two writers do.
 */
#ifndef HIMUON_H
#define HIMUON_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Storage type of every input and output matrix in a call. */
typedef enum himuon_dtype {
    HIMUON_F32 = 0,  /* IEEE binary32                                        */
    HIMUON_BF16 = 1  /* bfloat16; results rounded to nearest even on store   */
} himuon_dtype_t;

/* Operand type of the matrix-core (MFMA) products; accumulation, the
 * normalisation and the polynomial epilogues are fp32 in every mode. */
typedef enum himuon_compute {
    HIMUON_COMPUTE_DEFAULT = 0, /* F32 for f32 storage; for bf16 storage F16 when the
                                   coefficients keep every operand inside the fp16
                                   range (himuon_select_compute), else the call
                                   fails with HIMUON_ERR_RANGE (it never switches
                                   to BF16 operands on its own)                      */
    HIMUON_COMPUTE_F32 = 1,     /* fp32 operands (v_mfma_f32_32x32x2_f32)            */
    HIMUON_COMPUTE_F16 = 2,     /* fp16 operands, round-to-nearest-even              */
    HIMUON_COMPUTE_BF16 = 3     /* bf16 operands, round-to-nearest-even; fp32 range,
                                   but 8 significant bits: per-tile errors reach
                                   several 1e-2 at T <= 64 or K >= 8              */
} himuon_compute_t;

/* Status codes. Every error is detected before anything is enqueued: a call
 * that returns an error has left the stream and all buffers untouched. */
typedef enum himuon_status {
    HIMUON_OK = 0,
    HIMUON_ERR_INVALID_ARG = -1, /* null pointer, rows/cols < 1, ld < cols, K < 0,
                                    n_mats < 1, non-finite a/b/c, unknown enum     */
    HIMUON_ERR_UNSUPPORTED = -2, /* T not in {32, 64, 128, 256}, a dtype/compute
                                    pair that has no kernel, or (himuon_ns_tiled)
                                    2^32 or more tiles in one call                 */
    HIMUON_ERR_WORKSPACE = -3,   /* workspace smaller than the call's
                                    *_workspace_size, or a chunk budget smaller
                                    than one tile or problem                      */
    HIMUON_ERR_HIP = -4,         /* a HIP runtime call failed (see
                                    himuon_last_hip_error)                         */
    HIMUON_ERR_RANGE = -5        /* fp16 operands (HIMUON_COMPUTE_F16, or DEFAULT
                                    with bf16 storage) requested but the iterates
                                    can leave the fp16 range for these a, b, c, K  */
} himuon_status_t;

/* Device workspace bytes a himuon_ns_tiled call over n_mats matrices needs
 * when a fused tile kernel serves it (every T, dtype and compute mode except
 * the T = 256 calls below): the per-matrix descriptor table the kernels read
 * (64 bytes per matrix, rounded up to 256). Host-only; returns 0 for
 * n_mats < 1. */
size_t himuon_ns_tiled_workspace_size(int64_t n_mats);

/* Device workspace bytes of the himuon_ns_tiled call with these arguments,
 * whatever serves it: himuon_ns_tiled_workspace_size(n_mats) for a fused
 * kernel; for T = 256 with fp32 storage or bf16 operands, which have no fused
 * 256-tile kernel and run as 256 x 256 problems of the library-GEMM path
 * inside the same call, what himuon_ns_gemm_workspace_size gives for T = 256.
 * Host-only; 0 when the call would be rejected. */
size_t himuon_ns_tiled_call_workspace_size(int64_t n_mats, const int64_t* rows, const int64_t* cols, int T,
                                           int dtype, int compute, int K, float a, float b, float c,
                                           size_t chunk_budget_bytes);

/*
 * Y_l = Phi_{K,T}(X_l) for l = 0 .. n_mats-1, enqueued on `stream`.
 *
 * in_ptrs[l], out_ptrs[l]  device pointers to matrix l (storage `dtype`).
 *                          out_ptrs[l] == in_ptrs[l] (in place, same ld) is
 *                          allowed: each tile is read completely before any
 *                          of it is written, and one tile has one owner.
 *                          Any other overlap between matrices is undefined.
 * rows[l], cols[l]         H and W of matrix l (>= 1).
 * ld_in, ld_out            leading dimensions in elements (>= cols[l]); either
 *                          may be NULL, meaning contiguous rows (ld = cols).
 * T                        tile size, one of 32, 64, 128, 256. A matrix with
 *                          T >= max(H, W) is one zero-padded tile, which gives
 *                          Phi_K of the whole matrix (Sec. 4.4.3). T = 256 with
 *                          fp32 storage or bf16 operands has no fused kernel:
 *                          the call runs each 256-tile through the library
 *                          GEMMs of himuon_ns_gemm (same results up to
 *                          rounding; workspace and chunk budget as there).
 * K                        Newton-Schulz steps (>= 0). K = 0 returns S/||S||_F
 *                          per tile.
 * a, b, c                  the polynomial coefficients (finite), e.g. Muon's
 *                          quintic (3.4445, -4.7750, 2.0315), eq. (ns_quintic).
 * dtype, compute           himuon_dtype_t and himuon_compute_t values.
 * workspace                device memory of at least
 *                          himuon_ns_tiled_call_workspace_size(...) bytes (for a
 *                          fused kernel, himuon_ns_tiled_workspace_size(n_mats)),
 *                          owned by the caller; it must stay untouched until the
 *                          work enqueued by this call has completed on `stream`.
 * chunk_budget_bytes       bound on the bytes a chunk of tiles stands for
 *                          (input tile + output tile, 2*T*T*sizeof(dtype) per
 *                          tile); 0 means one chunk. Chunking never changes a
 *                          result bit.
 * stream                   hipStream_t to enqueue on.
 *
 * Returns HIMUON_OK once everything is enqueued (asynchronous: kernel faults
 * surface at the caller's next synchronisation). Non-finite input values stay
 * within their own tile. The host arrays are read only during the call; the
 * device buffers must outlive the enqueued work.
 */
int himuon_ns_tiled(int64_t n_mats,
                    const void* const* in_ptrs, void* const* out_ptrs,
                    const int64_t* rows, const int64_t* cols,
                    const int64_t* ld_in, const int64_t* ld_out,
                    int T, int K, float a, float b, float c,
                    int dtype, int compute,
                    void* workspace, size_t workspace_bytes,
                    size_t chunk_budget_bytes,
                    void* stream);

/*
 * himuon_ns_tiled with rectangular Th x Tw tiles in the fused kernels: each
 * matrix is padded to (R Th) x (C Tw), R = ceil(H/Th), C = ceil(W/Tw), every
 * tile goes through Phi_K on chip (one workgroup per tile, all K steps), and
 * a tile with Th > Tw is iterated as its transpose (the orientation rule of
 * Sec. 2.2, Phi_K(S) = Phi_K(S^T)^T), so the Gram matrix is the min(Th, Tw)
 * square one. This is the fused-kernel region of the tile-shape study
 * (Sec. 6.3, Th Tw <= 16384). Served shapes: {min(Th, Tw), max(Th, Tw)} in
 * {32} x {64, 128, 256} for fp32 storage (fp32 operands) and bf16 storage
 * (fp16 or bf16 operands), and {32} x {512}, {64} x {128, 256} for bf16
 * storage; both orientations of each;
 * Th = Tw is himuon_ns_tiled with T = Th. Other shapes return
 * HIMUON_ERR_UNSUPPORTED (himuon_ns_gemm_hw serves any shape on library
 * GEMMs). Arguments, workspace (himuon_ns_tiled_workspace_size(n_mats)),
 * chunk budget (2 Th Tw sizeof(dtype) bytes per tile), aliasing and errors as
 * himuon_ns_tiled.
 */
int himuon_ns_tiled_hw(int64_t n_mats,
                       const void* const* in_ptrs, void* const* out_ptrs,
                       const int64_t* rows, const int64_t* cols,
                       const int64_t* ld_in, const int64_t* ld_out,
                       int Th, int Tw, int K, float a, float b, float c,
                       int dtype, int compute,
                       void* workspace, size_t workspace_bytes,
                       size_t chunk_budget_bytes,
                       void* stream);

/* Most matrices one himuon_ns_tiled_noalloc call takes. */
#define HIMUON_NOALLOC_MAX_MATS 1024

/*
 * himuon_ns_tiled for callers that cannot allocate memory or own a workspace:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation. Same arguments, kernels, results (bit for bit) and errors as
 * himuon_ns_tiled, without workspace and workspace_bytes:
 *   - the per-matrix descriptor table lives in a 64 KiB device array that the
 *     library holds on each GPU it runs on until the process ends, so a call
 *     takes at most HIMUON_NOALLOC_MAX_MATS (1024) matrices; more is
 *     HIMUON_ERR_WORKSPACE, returned before anything is enqueued;
 *   - every call on a GPU of more than 32 matrices rewrites that array
 *     through small upload kernels enqueued on `stream` ahead of the tile
 *     kernels (smaller calls carry the table in the tile kernels' own
 *     arguments), so calls on one stream follow each other safely, but calls
 *     that overlap on one GPU (on different streams, or from several
 *     threads) race and must not be made;
 *   - the call allocates nothing, on the host or the device: no hipMalloc,
 *     no pinned staging; the descriptors travel in kernel arguments;
 *   - only calls a fused kernel serves: T = 256 with fp32 storage or bf16
 *     operands (the library-GEMM route, which needs a workspace) is
 *     HIMUON_ERR_UNSUPPORTED.
 */
int himuon_ns_tiled_noalloc(int64_t n_mats,
                            const void* const* in_ptrs, void* const* out_ptrs,
                            const int64_t* rows, const int64_t* cols,
                            const int64_t* ld_in, const int64_t* ld_out,
                            int T, int K, float a, float b, float c,
                            int dtype, int compute,
                            size_t chunk_budget_bytes,
                            void* stream);

/*
 * Phi_K through library GEMMs: the full-matrix branch and large tiles.
 *
 * T = 0: Phi_K of every whole matrix (the full-matrix branch, Sec. 4.4.3).
 *        A matrix with more rows than columns is worked on transposed,
 *        Phi_K(S) = Phi_K(S^T)^T, so the Gram matrix is min(H, W) square.
 * T >= 1: Phi_{K,T}, eq. (tiled_ns), with each T x T tile a problem of its
 *        own; meant for tiles too large to stay on one compute unit
 *        (T = 512 is the multi-kernel tile of Sec. 4.4.1), but any T works.
 *        A matrix with T >= max(H, W) is one whole problem as for T = 0
 *        (its single padded tile has the same Phi_K, Sec. 4.4.3).
 * Problems of equal shape are batched; each step of eq. (ns_iteration) is
 * three batched GEMMs (A = X X^T, B = bA + cA^2, X <- aX + BX) with fp32
 * accumulation. Operands are fp32 for fp32 storage; for bf16 storage fp16
 * (a rescaled iterate, himuon_select_compute's range argument applied to
 * the largest Gram size of the call) unless `compute` asks for bf16. The
 * norm of each problem is summed in fp64 in a fixed order, so a result does
 * not depend on the batch or chunk a problem lands in.
 *
 * Arguments are those of himuon_ns_tiled (out_ptrs[l] == in_ptrs[l] is
 * allowed: a chunk gathers all its blocks before it scatters any), except:
 * T                   0 or any positive tile size.
 * workspace           device memory of at least himuon_ns_gemm_workspace_size
 *                     (same arguments) bytes, owned by the caller: the
 *                     problem table, the iterate buffers of one chunk and
 *                     the GEMM library's scratch (64 MiB).
 * chunk_budget_bytes  bound on a chunk's iterate buffers (2 m n + 2 m^2
 *                     operand elements per problem); 0 = every problem of a
 *                     shape in one chunk (at most 65535).
 *
 * The first call on a device creates the GEMM library's handle there (its
 * own host and device resources, once per process); calls after that
 * allocate nothing. Errors as himuon_ns_tiled, plus HIMUON_ERR_UNSUPPORTED
 * when the GEMM library has no kernel for a shape or a Gram size exceeds
 * 32768.
 */
size_t himuon_ns_gemm_workspace_size(int64_t n_mats, const int64_t* rows, const int64_t* cols, int T,
                                     int dtype, int compute, int K, float a, float b, float c,
                                     size_t chunk_budget_bytes);

int himuon_ns_gemm(int64_t n_mats,
                   const void* const* in_ptrs, void* const* out_ptrs,
                   const int64_t* rows, const int64_t* cols,
                   const int64_t* ld_in, const int64_t* ld_out,
                   int T, int K, float a, float b, float c,
                   int dtype, int compute,
                   void* workspace, size_t workspace_bytes,
                   size_t chunk_budget_bytes,
                   void* stream);

/*
 * himuon_ns_gemm with rectangular Th x Tw tiles (the tile-shape study of
 * Sec. 6.3 and Sec. 2.1's tiling with T_h x T_w blocks): each matrix is padded
 * to (R Th) x (C Tw), R = ceil(H/Th), C = ceil(W/Tw), and every tile goes
 * through Phi_K, a tile with Th > Tw by the orientation rule (its transpose
 * is iterated, so the Gram matrix is min(Th, Tw) square). Th = Tw = T is
 * himuon_ns_gemm; Th = Tw = 0 is the full-matrix branch; exactly one of them
 * zero is HIMUON_ERR_INVALID_ARG. A matrix that one tile covers (Th >= H and
 * Tw >= W) is worked on whole. Other arguments, workspace and errors as
 * himuon_ns_gemm.
 */
size_t himuon_ns_gemm_hw_workspace_size(int64_t n_mats, const int64_t* rows, const int64_t* cols,
                                        int Th, int Tw, int dtype, int compute, int K,
                                        float a, float b, float c, size_t chunk_budget_bytes);

int himuon_ns_gemm_hw(int64_t n_mats,
                      const void* const* in_ptrs, void* const* out_ptrs,
                      const int64_t* rows, const int64_t* cols,
                      const int64_t* ld_in, const int64_t* ld_out,
                      int Th, int Tw, int K, float a, float b, float c,
                      int dtype, int compute,
                      void* workspace, size_t workspace_bytes,
                      size_t chunk_budget_bytes,
                      void* stream);

/*
 * Picks, for every GEMM that a himuon_ns_gemm (or GEMM-route himuon_step)
 * call with these shapes and arguments would run, the fastest of the GEMM
 * library's leading heuristic candidates (up to 8), by timing each on the
 * workspace's buffers on `stream`; later calls on this device use the
 * choice. Results never depend on it beyond the rounding of the GEMMs.
 *
 * Arguments as himuon_ns_gemm_workspace_size, plus workspace (at least that
 * many bytes; its contents are overwritten) and stream. Unlike the compute
 * entry points this call synchronises with `stream` (it waits on timing
 * events) and must not run concurrently with other calls on the device.
 * A shape set that was tuned before returns at once. Errors as
 * himuon_ns_gemm.
 */
int himuon_gemm_tune(int64_t n_mats, const int64_t* rows, const int64_t* cols, int T,
                     int dtype, int compute, int K, float a, float b, float c,
                     void* workspace, size_t workspace_bytes, size_t chunk_budget_bytes,
                     void* stream);

/* himuon_gemm_tune for the Th x Tw tilings of himuon_ns_gemm_hw. */
int himuon_gemm_tune_hw(int64_t n_mats, const int64_t* rows, const int64_t* cols, int Th, int Tw,
                        int dtype, int compute, int K, float a, float b, float c,
                        void* workspace, size_t workspace_bytes, size_t chunk_budget_bytes,
                        void* stream);

/*
 * One HiMuon optimizer step (Alg. 1) on n_mats parameter matrices, in place:
 *
 *   M_l <- beta M_l + G_l                            eq. (muon_momentum)
 *   Ghat = G_l + beta M_l  (nesterov != 0, eq. muon_lookahead), else M_l
 *   U    = Phi_K(Ghat)      if T = 0 (T = infinity) or T >= max(H_l, W_l),
 *          Phi_{K,T}(Ghat)  otherwise                 eq. (tiled_ns)
 *   W_l <- (1 - lr weight_decay) W_l - lr tau_l U     eq. (scaled_update)
 *   tau_l = scale_c sqrt(max(H_l, W_l)) on the full branch, scale_c sqrt(T)
 *           when tiled (Sec. 4.2; the paper's runs use scale_c = 0.2).
 *
 * weights[l], grads[l], moms[l]  device pointers, storage `dtype`, one
 *                          row-major layout (leading dimension ld[l]; ld may
 *                          be NULL for contiguous rows). W and M are updated in
 *                          place; G is only read. The three must not overlap
 *                          (equal pointers are rejected). The new M is stored
 *                          rounded to `dtype`, and the lookahead is formed from
 *                          the stored value.
 * T, K, a, b, c            as himuon_ns_gemm: T = 0 or any positive tile size.
 *                          Routes: T in {32, 64, 128} runs the step inside the
 *                          fused tile kernel (fp32 storage, bf16 operands, or
 *                          fp16 operands with c > 0; U is rounded to `dtype`
 *                          before the update, and with fp16 operands so is the
 *                          lookahead as the tile is staged); T = 256, and fp16
 *                          operands with c <= 0, run an element-wise prologue
 *                          and epilogue around the fused kernel, with the
 *                          lookahead held in `dtype` in the workspace; any
 *                          other T runs the library-GEMM path with the
 *                          momentum fused into its gather and the update into
 *                          its scatter.
 * lr, momentum, weight_decay, nesterov, scale_c   the step's scalars (finite).
 * workspace                device memory of at least himuon_step_workspace_size
 *                          (same arguments) bytes, owned by the caller.
 * chunk_budget_bytes       in-kernel route: as himuon_ns_tiled; prologue and
 *                          epilogue route: bound on the lookahead buffers of
 *                          one group of consecutive matrices (0: one group);
 *                          GEMM route: as himuon_ns_gemm.
 *
 * Errors as himuon_ns_gemm; nothing is enqueued when one is returned.
 * Matrices with non-finite gradients or momenta give non-finite weights
 * only within their own problems (tiles or whole matrix).
 */
size_t himuon_step_workspace_size(int64_t n_mats, const int64_t* rows, const int64_t* cols, int T,
                                  int dtype, int compute, int K, float a, float b, float c,
                                  size_t chunk_budget_bytes);

int himuon_step(int64_t n_mats,
                void* const* weights, const void* const* grads, void* const* moms,
                const int64_t* rows, const int64_t* cols, const int64_t* ld,
                int T, int K, float a, float b, float c,
                float lr, float momentum, float weight_decay, int nesterov, float scale_c,
                int dtype, int compute,
                void* workspace, size_t workspace_bytes,
                size_t chunk_budget_bytes,
                void* stream);

/*
 * Plans: a himuon_ns_tiled, himuon_ns_gemm or himuon_step call recorded
 * once, on the current device, into a HIP graph and replayed by
 * himuon_plan_launch, whose only host work is one graph launch (no
 * validation, planning or table staging per call, and one launch for the
 * whole chain of kernels of a library-GEMM call). This is the graph-captured
 * cross-layer optimizer step of the optimizer-step study (Sec. 6.4) and the
 * graph-capture state that the runtime tile-size reconfiguration rebuilds
 * when T changes (Sec. 4.4.3).
 *
 * himuon_plan_ns_tiled / himuon_plan_ns_gemm / himuon_plan_step take the
 * arguments of himuon_ns_tiled / himuon_ns_gemm / himuon_step without the
 * stream, validate them as those do (returning the same errors, with
 * *plan = NULL), and record the call:
 * every device pointer and every scalar is fixed in the plan. Each launch
 * then performs the recorded call again on the current contents of those
 * buffers, in `stream` order: it first copies the call's descriptor tables
 * from pinned host buffers that the plan owns into `workspace`, so the
 * workspace and every matrix must stay allocated, and the workspace must not
 * be used by other work that overlaps a launch, until the plan is destroyed.
 * A launch's results equal those of the recorded call bit for bit.
 * Recording synchronises nothing and enqueues nothing on the caller's
 * streams; it allocates the plan's host memory, a private stream and the
 * graph (configuration-time calls, like himuon_gemm_tune).
 *
 * himuon_plan_launch returns HIMUON_ERR_INVALID_ARG for a NULL plan or a
 * stream on another device than the plan's; himuon_plan_destroy frees the
 * plan (NULL is a no-op) and must not be called while a launch of it may
 * still run.
 */
typedef struct himuon_plan himuon_plan_t;

int himuon_plan_ns_tiled(himuon_plan_t** plan, int64_t n_mats,
                         const void* const* in_ptrs, void* const* out_ptrs,
                         const int64_t* rows, const int64_t* cols,
                         const int64_t* ld_in, const int64_t* ld_out,
                         int T, int K, float a, float b, float c,
                         int dtype, int compute,
                         void* workspace, size_t workspace_bytes,
                         size_t chunk_budget_bytes);

int himuon_plan_ns_gemm(himuon_plan_t** plan, int64_t n_mats,
                        const void* const* in_ptrs, void* const* out_ptrs,
                        const int64_t* rows, const int64_t* cols,
                        const int64_t* ld_in, const int64_t* ld_out,
                        int T, int K, float a, float b, float c,
                        int dtype, int compute,
                        void* workspace, size_t workspace_bytes,
                        size_t chunk_budget_bytes);

int himuon_plan_step(himuon_plan_t** plan, int64_t n_mats,
                     void* const* weights, const void* const* grads, void* const* moms,
                     const int64_t* rows, const int64_t* cols, const int64_t* ld,
                     int T, int K, float a, float b, float c,
                     float lr, float momentum, float weight_decay, int nesterov, float scale_c,
                     int dtype, int compute,
                     void* workspace, size_t workspace_bytes,
                     size_t chunk_budget_bytes);

int himuon_plan_launch(const himuon_plan_t* plan, void* stream);

void himuon_plan_destroy(himuon_plan_t* plan);

/*
 * Host-only planner (no HIP call): the tiles and chunks himuon_ns_tiled
 * would use, i.e. the memory-bounded chunking of cross-layer batches of
 * Sec. 4.4.2 (a batch larger than the memory budget is split into the
 * fewest chunks that fit). Tiles are numbered matrix by matrix, row-major over each
 * matrix's R x C grid. The chunk count is the fewest whose per-chunk bytes
 * (2*T*T*sizeof(dtype) per tile) fit chunk_budget_bytes (0: one chunk), and
 * the chunks are balanced: chunk i covers [bounds[i], bounds[i+1]) with
 * sizes that differ by at most one tile.
 *
 * T may be any value >= 1 here (planning only). *total_tiles and *n_chunks
 * are always written on success; chunk_bounds (may be NULL) receives
 * n_chunks + 1 entries when max_bounds >= n_chunks + 1.
 * Errors: HIMUON_ERR_INVALID_ARG, HIMUON_ERR_WORKSPACE (budget below one tile).
 */
int himuon_plan_chunks(int64_t n_mats, const int64_t* rows, const int64_t* cols,
                       int T, int dtype, size_t chunk_budget_bytes,
                       int64_t* total_tiles, int64_t* n_chunks,
                       int64_t* chunk_bounds, int64_t max_bounds);

/*
 * Host-only: the compute mode a call with these arguments resolves to
 * (a himuon_compute_t value >= 1), or a negative status. For bf16 storage
 * and HIMUON_COMPUTE_DEFAULT it returns F16 when the scalar iterates
 * p^k(s), s in [0, 1], k <= K (p(s) = as + bs^3 + cs^5, which is what every
 * singular value of the normalised tile follows, Sec. 2.2) bound |X|, |A|,
 * |A^2| and |bA + cA^2| well inside fp16's range, else HIMUON_ERR_RANGE.
 */
int himuon_select_compute(int dtype, int compute, int K, float a, float b, float c);

/* Static English text for a status code. */
const char* himuon_status_string(int status);

/* The hipError_t value behind the calling thread's last HIMUON_ERR_HIP. */
int himuon_last_hip_error(void);

/* Library version, major*10000 + minor*100 + patch. */
int himuon_version(void);

/*
 * Measurement aid, not part of the map: a launch that runs nothing but dense
 * 32x32x16 MFMA products (fp16 operands for compute = HIMUON_COMPUTE_F16,
 * bf16 for HIMUON_COMPUTE_BF16, fp32 accumulation), the ceiling against which
 * the roofline of the tile kernels' issued MFMA work is read. `grid`
 * workgroups of 256 threads; every wave issues 4 * iters products with four
 * independent accumulators, so one launch performs
 *     grid * 4 * 4 * iters * 32 * 32 * 16 * 2   flops.
 * ops: device memory of 4096 16-byte words (64 KiB) of operand bits, read
 * only (read once per lane). out: device memory of grid * 256 floats,
 * written (the lanes' sums, so that nothing is optimised away). Enqueue only,
 * on `stream` (NULL: the default stream). Errors: HIMUON_ERR_INVALID_ARG
 * (null pointer, grid or iters below 1, grid above 2^20, another compute
 * value),
 * HIMUON_ERR_HIP.
 */
int himuon_calib_mfma(int compute, const void* ops, float* out, int grid, int iters, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HIMUON_H */
