"""Python binding of libhimuon.so, the MI355X tiled Newton–Schulz library.

Argument marshalling only: every step of the map (tiling, normalisation, the
K Newton–Schulz steps, reassembly, batching and chunking) runs in the native
library declared in ``include/himuon.h``. PyTorch is used for device memory
and streams. If the library is missing the import of any entry point raises;
there is no fallback implementation.

Low-level names mirror the C ABI (``himuon_ns_tiled``, ``himuon_plan_chunks``,
``himuon_ns_tiled_workspace_size``, ``himuon_select_compute``,
``himuon_status_string``, ``himuon_last_hip_error``, ``himuon_version``);
``ns_tiled`` is the tensor-level convenience wrapper.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(PKG, "libhimuon.so")

# himuon_dtype_t / himuon_compute_t / himuon_status_t
F32, BF16 = 0, 1
COMPUTE_DEFAULT, COMPUTE_F32, COMPUTE_F16, COMPUTE_BF16 = 0, 1, 2, 3
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_RANGE = 0, -1, -2, -3, -4, -5
TILE_SIZES = (32, 64, 128, 256)
QUINTIC = (3.4445, -4.7750, 2.0315)  # eq. (ns_quintic)

_lib = None


class HimuonError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        msg = f"{what}: {himuon_status_string(status)} (status {status})"
        if status == ERR_HIP:
            msg += f", hipError {himuon_last_hip_error()}"
        super().__init__(msg)


def lib():
    """The loaded native library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            raise ImportError(f"{LIBRARY} is missing; build it with "
                              "`python -m paper_2606_27216_amd.build_lib`")
        L = ctypes.CDLL(LIBRARY)
        i64, vp, sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t
        L.himuon_ns_tiled_workspace_size.argtypes = [i64]
        L.himuon_ns_tiled_workspace_size.restype = sz
        L.himuon_ns_tiled_call_workspace_size.argtypes = [i64, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                          ctypes.c_int, ctypes.c_float, ctypes.c_float,
                                                          ctypes.c_float, sz]
        L.himuon_ns_tiled_call_workspace_size.restype = sz
        L.himuon_ns_tiled.argtypes = [i64, vp, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                      ctypes.c_int, ctypes.c_int, vp, sz, sz, vp]
        L.himuon_ns_tiled.restype = ctypes.c_int
        L.himuon_ns_tiled_hw.argtypes = [i64, vp, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                         ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_int, ctypes.c_int,
                                         vp, sz, sz, vp]
        L.himuon_ns_tiled_hw.restype = ctypes.c_int
        L.himuon_ns_tiled_noalloc.argtypes = [i64, vp, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int,
                                              ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                              ctypes.c_int, ctypes.c_int, sz, vp]
        L.himuon_ns_tiled_noalloc.restype = ctypes.c_int
        L.himuon_ns_gemm_workspace_size.argtypes = [i64, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                    ctypes.c_int, ctypes.c_float, ctypes.c_float,
                                                    ctypes.c_float, sz]
        L.himuon_ns_gemm_workspace_size.restype = sz
        L.himuon_ns_gemm.argtypes = L.himuon_ns_tiled.argtypes
        L.himuon_ns_gemm.restype = ctypes.c_int
        L.himuon_step_workspace_size.argtypes = L.himuon_ns_gemm_workspace_size.argtypes
        L.himuon_step_workspace_size.restype = sz
        f = ctypes.c_float
        L.himuon_step.argtypes = [i64, vp, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int, f, f, f,
                                  f, f, f, ctypes.c_int, f, ctypes.c_int, ctypes.c_int, vp, sz, sz, vp]
        L.himuon_step.restype = ctypes.c_int
        L.himuon_gemm_tune.argtypes = [i64, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       f, f, f, vp, sz, sz, vp]
        L.himuon_gemm_tune.restype = ctypes.c_int
        L.himuon_gemm_tune_hw.argtypes = [i64, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_int, f, f, f, vp, sz, sz, vp]
        L.himuon_gemm_tune_hw.restype = ctypes.c_int
        L.himuon_ns_gemm_hw_workspace_size.argtypes = [i64, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                       ctypes.c_int, ctypes.c_int, f, f, f, sz]
        L.himuon_ns_gemm_hw_workspace_size.restype = sz
        L.himuon_ns_gemm_hw.argtypes = [i64, vp, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                        f, f, f, ctypes.c_int, ctypes.c_int, vp, sz, sz, vp]
        L.himuon_ns_gemm_hw.restype = ctypes.c_int
        L.himuon_plan_ns_tiled.argtypes = [vp, i64, vp, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int,
                                           f, f, f, ctypes.c_int, ctypes.c_int, vp, sz, sz]
        L.himuon_plan_ns_tiled.restype = ctypes.c_int
        L.himuon_plan_ns_gemm.argtypes = [vp, i64, vp, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int,
                                          f, f, f, ctypes.c_int, ctypes.c_int, vp, sz, sz]
        L.himuon_plan_ns_gemm.restype = ctypes.c_int
        L.himuon_plan_step.argtypes = [vp, i64, vp, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int, f, f, f,
                                       f, f, f, ctypes.c_int, f, ctypes.c_int, ctypes.c_int, vp, sz, sz]
        L.himuon_plan_step.restype = ctypes.c_int
        L.himuon_plan_launch.argtypes = [vp, vp]
        L.himuon_plan_launch.restype = ctypes.c_int
        L.himuon_plan_destroy.argtypes = [vp]
        L.himuon_plan_destroy.restype = None
        L.himuon_plan_chunks.argtypes = [i64, vp, vp, ctypes.c_int, ctypes.c_int, sz, vp, vp, vp, i64]
        L.himuon_plan_chunks.restype = ctypes.c_int
        L.himuon_select_compute.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                            ctypes.c_float, ctypes.c_float, ctypes.c_float]
        L.himuon_select_compute.restype = ctypes.c_int
        L.himuon_status_string.argtypes = [ctypes.c_int]
        L.himuon_status_string.restype = ctypes.c_char_p
        L.himuon_last_hip_error.argtypes = []
        L.himuon_last_hip_error.restype = ctypes.c_int
        L.himuon_version.argtypes = []
        L.himuon_version.restype = ctypes.c_int
        L.himuon_calib_mfma.argtypes = [ctypes.c_int, vp, vp, ctypes.c_int, ctypes.c_int, vp]
        L.himuon_calib_mfma.restype = ctypes.c_int
        _lib = L
    return _lib


def _i64_array(vals):
    vals = [int(v) for v in vals]
    return (ctypes.c_int64 * len(vals))(*vals)


def _ptr_array(vals):
    vals = [int(v) for v in vals]
    return (ctypes.c_void_p * len(vals))(*vals)


# ---------------------------------------------------------------- raw C ABI

def himuon_ns_tiled_workspace_size(n_mats: int) -> int:
    return int(lib().himuon_ns_tiled_workspace_size(int(n_mats)))


def himuon_ns_tiled_call_workspace_size(rows, cols, T, dtype, compute, K, a, b, c, chunk_budget_bytes=0) -> int:
    """Workspace bytes of the himuon_ns_tiled call with these arguments (0 if it would be rejected)."""
    return int(lib().himuon_ns_tiled_call_workspace_size(
        len(rows), _i64_array(rows), _i64_array(cols), int(T), int(dtype), int(compute), int(K),
        float(a), float(b), float(c), int(chunk_budget_bytes)))


def himuon_ns_tiled(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, T, K, a, b, c,
                    dtype, compute, workspace, workspace_bytes, chunk_budget_bytes, stream) -> int:
    """Same arguments as the C function; Python sequences for the per-matrix
    arrays (``ld_in``/``ld_out`` may be None), integers for device pointers
    and the stream handle. Returns the status code."""
    return int(lib().himuon_ns_tiled(
        int(n_mats), _ptr_array(in_ptrs), _ptr_array(out_ptrs), _i64_array(rows), _i64_array(cols),
        None if ld_in is None else _i64_array(ld_in), None if ld_out is None else _i64_array(ld_out),
        int(T), int(K), float(a), float(b), float(c), int(dtype), int(compute),
        int(workspace) if workspace else None, int(workspace_bytes), int(chunk_budget_bytes),
        int(stream) if stream else None))


def himuon_ns_tiled_hw(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, Th, Tw, K, a, b, c,
                       dtype, compute, workspace, workspace_bytes, chunk_budget_bytes, stream) -> int:
    """Same arguments as the C function (see himuon_ns_tiled). Returns the status code."""
    return int(lib().himuon_ns_tiled_hw(
        int(n_mats), _ptr_array(in_ptrs), _ptr_array(out_ptrs), _i64_array(rows), _i64_array(cols),
        None if ld_in is None else _i64_array(ld_in), None if ld_out is None else _i64_array(ld_out),
        int(Th), int(Tw), int(K), float(a), float(b), float(c), int(dtype), int(compute),
        int(workspace) if workspace else None, int(workspace_bytes), int(chunk_budget_bytes),
        int(stream) if stream else None))


NOALLOC_MAX_MATS = 1024  # HIMUON_NOALLOC_MAX_MATS


def himuon_ns_tiled_noalloc(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, T, K, a, b, c,
                            dtype, compute, chunk_budget_bytes, stream) -> int:
    """Same arguments as the C function (himuon_ns_tiled without the
    workspace). Returns the status code."""
    return int(lib().himuon_ns_tiled_noalloc(
        int(n_mats), _ptr_array(in_ptrs), _ptr_array(out_ptrs), _i64_array(rows), _i64_array(cols),
        None if ld_in is None else _i64_array(ld_in), None if ld_out is None else _i64_array(ld_out),
        int(T), int(K), float(a), float(b), float(c), int(dtype), int(compute), int(chunk_budget_bytes),
        int(stream) if stream else None))


def himuon_ns_gemm_workspace_size(rows, cols, T, dtype, compute, K, a, b, c, chunk_budget_bytes=0) -> int:
    """Workspace bytes of a himuon_ns_gemm call over matrices of these shapes (0 on an invalid plan)."""
    return int(lib().himuon_ns_gemm_workspace_size(
        len(rows), _i64_array(rows), _i64_array(cols), int(T), int(dtype), int(compute), int(K),
        float(a), float(b), float(c), int(chunk_budget_bytes)))


def himuon_ns_gemm(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, T, K, a, b, c,
                   dtype, compute, workspace, workspace_bytes, chunk_budget_bytes, stream) -> int:
    """Same arguments as the C function (see himuon_ns_tiled). Returns the status code."""
    return int(lib().himuon_ns_gemm(
        int(n_mats), _ptr_array(in_ptrs), _ptr_array(out_ptrs), _i64_array(rows), _i64_array(cols),
        None if ld_in is None else _i64_array(ld_in), None if ld_out is None else _i64_array(ld_out),
        int(T), int(K), float(a), float(b), float(c), int(dtype), int(compute),
        int(workspace) if workspace else None, int(workspace_bytes), int(chunk_budget_bytes),
        int(stream) if stream else None))


def himuon_step_workspace_size(rows, cols, T, dtype, compute, K, a, b, c, chunk_budget_bytes=0) -> int:
    """Workspace bytes of a himuon_step call over matrices of these shapes (0 on an invalid plan)."""
    return int(lib().himuon_step_workspace_size(
        len(rows), _i64_array(rows), _i64_array(cols), int(T), int(dtype), int(compute), int(K),
        float(a), float(b), float(c), int(chunk_budget_bytes)))


def himuon_step(n_mats, weights, grads, moms, rows, cols, ld, T, K, a, b, c, lr, momentum, weight_decay,
                nesterov, scale_c, dtype, compute, workspace, workspace_bytes, chunk_budget_bytes, stream) -> int:
    """Same arguments as the C function (``ld`` may be None). Returns the status code."""
    return int(lib().himuon_step(
        int(n_mats), _ptr_array(weights), _ptr_array(grads), _ptr_array(moms), _i64_array(rows),
        _i64_array(cols), None if ld is None else _i64_array(ld), int(T), int(K), float(a), float(b),
        float(c), float(lr), float(momentum), float(weight_decay), int(bool(nesterov)), float(scale_c),
        int(dtype), int(compute), int(workspace) if workspace else None, int(workspace_bytes),
        int(chunk_budget_bytes), int(stream) if stream else None))


def himuon_ns_gemm_hw_workspace_size(rows, cols, Th, Tw, dtype, compute, K, a, b, c, chunk_budget_bytes=0) -> int:
    """Workspace bytes of a himuon_ns_gemm_hw call (0 on an invalid plan)."""
    return int(lib().himuon_ns_gemm_hw_workspace_size(
        len(rows), _i64_array(rows), _i64_array(cols), int(Th), int(Tw), int(dtype), int(compute), int(K),
        float(a), float(b), float(c), int(chunk_budget_bytes)))


def himuon_ns_gemm_hw(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, Th, Tw, K, a, b, c,
                      dtype, compute, workspace, workspace_bytes, chunk_budget_bytes, stream) -> int:
    """Same arguments as the C function (see himuon_ns_tiled). Returns the status code."""
    return int(lib().himuon_ns_gemm_hw(
        int(n_mats), _ptr_array(in_ptrs), _ptr_array(out_ptrs), _i64_array(rows), _i64_array(cols),
        None if ld_in is None else _i64_array(ld_in), None if ld_out is None else _i64_array(ld_out),
        int(Th), int(Tw), int(K), float(a), float(b), float(c), int(dtype), int(compute),
        int(workspace) if workspace else None, int(workspace_bytes), int(chunk_budget_bytes),
        int(stream) if stream else None))


def himuon_gemm_tune_hw(rows, cols, Th, Tw, dtype, compute, K, a, b, c, workspace, workspace_bytes,
                        chunk_budget_bytes=0, stream=None) -> int:
    """Same arguments as the C function. Returns the status code."""
    return int(lib().himuon_gemm_tune_hw(
        len(rows), _i64_array(rows), _i64_array(cols), int(Th), int(Tw), int(dtype), int(compute), int(K),
        float(a), float(b), float(c), int(workspace) if workspace else None, int(workspace_bytes),
        int(chunk_budget_bytes), int(stream) if stream else None))


def himuon_gemm_tune(rows, cols, T, dtype, compute, K, a, b, c, workspace, workspace_bytes,
                     chunk_budget_bytes=0, stream=None) -> int:
    """Same arguments as the C function (``workspace`` a device pointer). Returns the status code."""
    return int(lib().himuon_gemm_tune(
        len(rows), _i64_array(rows), _i64_array(cols), int(T), int(dtype), int(compute), int(K),
        float(a), float(b), float(c), int(workspace) if workspace else None, int(workspace_bytes),
        int(chunk_budget_bytes), int(stream) if stream else None))


def gemm_tune(shapes, T, dtype, K=5, coeffs=QUINTIC, compute=COMPUTE_DEFAULT, chunk_budget_bytes=0,
              workspace=None, stream=None, device="cuda", Tw=None):
    """Time the GEMM library's candidates for the GEMM-path calls over matrices
    of these ``(rows, cols)`` shapes (T = 0, square T x T tiles, or T x Tw
    tiles) and keep the fastest; synchronises. ``dtype`` is F32 or BF16."""
    import torch
    a, b, c = coeffs
    Th, Tw = int(T), int(T if Tw is None else Tw)
    rows = [int(h) for h, _ in shapes]
    cols = [int(w) for _, w in shapes]
    need = himuon_ns_gemm_hw_workspace_size(rows, cols, Th, Tw, dtype, compute, K, a, b, c, chunk_budget_bytes)
    if need == 0:
        raise HimuonError(ERR_INVALID_ARG, "himuon_ns_gemm_hw_workspace_size")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    if stream is None:
        stream = torch.cuda.current_stream(workspace.device)
    st = himuon_gemm_tune_hw(rows, cols, Th, Tw, dtype, compute, K, a, b, c, workspace.data_ptr(),
                             workspace.numel() * workspace.element_size(), chunk_budget_bytes, stream.cuda_stream)
    if st != OK:
        raise HimuonError(st, "himuon_gemm_tune_hw")


def himuon_plan_ns_tiled(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, T, K, a, b, c, dtype, compute,
                         workspace, workspace_bytes, chunk_budget_bytes):
    """Records a himuon_ns_tiled call into a plan. Returns (status, plan handle or None)."""
    h = ctypes.c_void_p()
    st = int(lib().himuon_plan_ns_tiled(
        ctypes.byref(h), int(n_mats), _ptr_array(in_ptrs), _ptr_array(out_ptrs), _i64_array(rows), _i64_array(cols),
        None if ld_in is None else _i64_array(ld_in), None if ld_out is None else _i64_array(ld_out),
        int(T), int(K), float(a), float(b), float(c), int(dtype), int(compute),
        int(workspace) if workspace else None, int(workspace_bytes), int(chunk_budget_bytes)))
    return st, (h.value if st == OK else None)


def himuon_plan_ns_gemm(n_mats, in_ptrs, out_ptrs, rows, cols, ld_in, ld_out, T, K, a, b, c, dtype, compute,
                        workspace, workspace_bytes, chunk_budget_bytes):
    """Records a himuon_ns_gemm call into a plan. Returns (status, plan handle or None)."""
    h = ctypes.c_void_p()
    st = int(lib().himuon_plan_ns_gemm(
        ctypes.byref(h), int(n_mats), _ptr_array(in_ptrs), _ptr_array(out_ptrs), _i64_array(rows), _i64_array(cols),
        None if ld_in is None else _i64_array(ld_in), None if ld_out is None else _i64_array(ld_out),
        int(T), int(K), float(a), float(b), float(c), int(dtype), int(compute),
        int(workspace) if workspace else None, int(workspace_bytes), int(chunk_budget_bytes)))
    return st, (h.value if st == OK else None)


def himuon_plan_step(n_mats, weights, grads, moms, rows, cols, ld, T, K, a, b, c, lr, momentum, weight_decay,
                     nesterov, scale_c, dtype, compute, workspace, workspace_bytes, chunk_budget_bytes):
    """Records a himuon_step call into a plan. Returns (status, plan handle or None)."""
    h = ctypes.c_void_p()
    st = int(lib().himuon_plan_step(
        ctypes.byref(h), int(n_mats), _ptr_array(weights), _ptr_array(grads), _ptr_array(moms), _i64_array(rows),
        _i64_array(cols), None if ld is None else _i64_array(ld), int(T), int(K), float(a), float(b), float(c),
        float(lr), float(momentum), float(weight_decay), int(bool(nesterov)), float(scale_c), int(dtype),
        int(compute), int(workspace) if workspace else None, int(workspace_bytes), int(chunk_budget_bytes)))
    return st, (h.value if st == OK else None)


def himuon_plan_launch(plan, stream) -> int:
    return int(lib().himuon_plan_launch(plan, int(stream) if stream else None))


def himuon_plan_destroy(plan) -> None:
    lib().himuon_plan_destroy(plan)


class Plan:
    """A recorded call (``himuon_plan_*``): ``launch(stream)`` replays it.
    Keeps the tensors it was recorded on (and its workspace) alive."""

    def __init__(self, handle, keep):
        self.handle = handle
        self._keep = keep

    def launch(self, stream=None):
        import torch
        if stream is None:
            stream = torch.cuda.current_stream()
        st = himuon_plan_launch(self.handle, stream.cuda_stream)
        if st != OK:
            raise HimuonError(st, "himuon_plan_launch")

    def close(self):
        if self.handle:
            import torch
            torch.cuda.synchronize()
            himuon_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def plan_ns_tiled(inputs, outputs, T=128, K=5, coeffs=QUINTIC, compute=COMPUTE_DEFAULT, chunk_budget_bytes=0,
                  workspace=None):
    """Records ``ns_tiled(inputs, outputs, ...)`` into a Plan (on the inputs'
    device); every launch recomputes the outputs from the inputs' current
    contents."""
    import torch
    inputs, outputs = list(inputs), list(outputs)
    code = _dtype_code(inputs[0])
    dev = inputs[0].device
    a, b, c = coeffs
    rows = [x.shape[0] for x in inputs]
    cols = [x.shape[1] for x in inputs]
    if workspace is None:
        need = himuon_ns_tiled_call_workspace_size(rows, cols, T, code, compute, K, a, b, c, chunk_budget_bytes)
        workspace = torch.empty(max(need, himuon_ns_tiled_workspace_size(len(inputs))), dtype=torch.uint8,
                                device=dev)
    with torch.cuda.device(dev):
        st, h = himuon_plan_ns_tiled(
            len(inputs), [x.data_ptr() for x in inputs], [y.data_ptr() for y in outputs], rows, cols,
            [x.stride(0) for x in inputs], [y.stride(0) for y in outputs], T, K, a, b, c, code, compute,
            workspace.data_ptr(), workspace.numel() * workspace.element_size(), chunk_budget_bytes)
    if st != OK:
        raise HimuonError(st, "himuon_plan_ns_tiled")
    return Plan(h, (inputs, outputs, workspace))


def plan_ns_gemm(inputs, outputs, T=0, K=5, coeffs=QUINTIC, compute=COMPUTE_DEFAULT, chunk_budget_bytes=0,
                 workspace=None):
    """Records ``ns_gemm(inputs, outputs, ...)`` (square T x T tiles, or whole
    matrices for T = 0) into a Plan on the inputs' device; every launch
    recomputes the outputs from the inputs' current contents."""
    import torch
    inputs, outputs = list(inputs), list(outputs)
    code = _dtype_code(inputs[0])
    dev = inputs[0].device
    a, b, c = coeffs
    rows = [x.shape[0] for x in inputs]
    cols = [x.shape[1] for x in inputs]
    if workspace is None:
        need = himuon_ns_gemm_workspace_size(rows, cols, T, code, compute, K, a, b, c, chunk_budget_bytes)
        if need == 0:
            raise HimuonError(ERR_INVALID_ARG, "himuon_ns_gemm_workspace_size")
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    with torch.cuda.device(dev):
        st, h = himuon_plan_ns_gemm(
            len(inputs), [x.data_ptr() for x in inputs], [y.data_ptr() for y in outputs], rows, cols,
            [x.stride(0) for x in inputs], [y.stride(0) for y in outputs], T, K, a, b, c, code, compute,
            workspace.data_ptr(), workspace.numel() * workspace.element_size(), chunk_budget_bytes)
    if st != OK:
        raise HimuonError(st, "himuon_plan_ns_gemm")
    return Plan(h, (inputs, outputs, workspace))


def himuon_plan_chunks(rows, cols, T, dtype=BF16, chunk_budget_bytes=0):
    """Returns (total_tiles, [chunk bounds]) or raises HimuonError."""
    n = len(rows)
    total = ctypes.c_int64()
    nch = ctypes.c_int64()
    st = lib().himuon_plan_chunks(n, _i64_array(rows), _i64_array(cols), int(T), int(dtype),
                                  int(chunk_budget_bytes), ctypes.byref(total), ctypes.byref(nch), None, 0)
    if st != OK:
        raise HimuonError(st, "himuon_plan_chunks")
    bounds = (ctypes.c_int64 * (nch.value + 1))()
    st = lib().himuon_plan_chunks(n, _i64_array(rows), _i64_array(cols), int(T), int(dtype),
                                  int(chunk_budget_bytes), ctypes.byref(total), ctypes.byref(nch),
                                  bounds, nch.value + 1)
    if st != OK:
        raise HimuonError(st, "himuon_plan_chunks")
    return total.value, list(bounds)


def himuon_select_compute(dtype, compute, K, a, b, c) -> int:
    return int(lib().himuon_select_compute(int(dtype), int(compute), int(K), float(a), float(b), float(c)))


def himuon_status_string(status: int) -> str:
    return lib().himuon_status_string(int(status)).decode()


def himuon_last_hip_error() -> int:
    return int(lib().himuon_last_hip_error())


def himuon_version() -> int:
    return int(lib().himuon_version())


def himuon_calib_mfma(compute: int, ops: int, out: int, grid: int, iters: int, stream: int = 0) -> int:
    return int(lib().himuon_calib_mfma(compute, ops, out, grid, iters, stream))


# ------------------------------------------------------------ tensor wrapper

def _keep_alive(tensors, stream, dev):
    """Tensors this module allocated for a call enqueued on ``stream``: when
    that is not torch's current stream, tell the caching allocator that
    ``stream`` uses them, so that their memory is not handed out again
    before the enqueued work has finished."""
    import torch
    if stream != torch.cuda.current_stream(dev):
        for t in tensors:
            t.record_stream(stream)


def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}; expected float32 or bfloat16")


def ns_tiled(inputs, outputs=None, T=128, K=5, coeffs=QUINTIC, compute=COMPUTE_DEFAULT,
             chunk_budget_bytes=0, workspace=None, stream=None, Tw=None):
    """Φ_{K,T} of every 2-D CUDA tensor in ``inputs`` in one library call
    (with ``Tw``: rectangular T x Tw tiles, himuon_ns_tiled_hw).

    ``outputs`` defaults to fresh tensors; passing ``outputs=inputs`` runs in
    place. Rows may be strided (``stride(1) == 1`` is required). The call is
    asynchronous on ``stream`` (default: torch's current stream). Returns the
    outputs."""
    import torch
    inputs = list(inputs)
    if not inputs:
        raise ValueError("no matrices")
    code = _dtype_code(inputs[0])
    dev = inputs[0].device
    for x in inputs:
        if x.dim() != 2 or not x.is_cuda or x.device != dev or _dtype_code(x) != code or x.stride(1) != 1:
            raise ValueError("inputs must be 2-D row-major CUDA tensors of one dtype on one device")
    fresh = []  # tensors allocated here for the call
    if outputs is None:
        outputs = [torch.empty_like(x, memory_format=torch.contiguous_format) for x in inputs]
        fresh += outputs
    outputs = list(outputs)
    if len(outputs) != len(inputs):
        raise ValueError("inputs and outputs differ in length")
    for x, y in zip(inputs, outputs):
        if y.shape != x.shape or y.dtype != x.dtype or y.device != dev or y.stride(1) != 1:
            raise ValueError("each output must match its input's shape, dtype and device")
    n = len(inputs)
    a, b, c = coeffs
    rows = [x.shape[0] for x in inputs]
    cols = [x.shape[1] for x in inputs]
    if workspace is None:
        need = 0 if Tw is not None and Tw != T else \
            himuon_ns_tiled_call_workspace_size(rows, cols, T, code, compute, K, a, b, c, chunk_budget_bytes)
        # (a call that would be rejected still gets a table-sized workspace, so
        # that the library reports the precise error)
        workspace = torch.empty(max(need, himuon_ns_tiled_workspace_size(n)), dtype=torch.uint8, device=dev)
        fresh.append(workspace)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    ptrs = ([x.data_ptr() for x in inputs], [y.data_ptr() for y in outputs], rows, cols,
            [x.stride(0) for x in inputs], [y.stride(0) for y in outputs])
    ws = (workspace.data_ptr(), workspace.numel() * workspace.element_size(), chunk_budget_bytes, stream.cuda_stream)
    if Tw is None or Tw == T:
        st = himuon_ns_tiled(n, *ptrs, T, K, a, b, c, code, compute, *ws)
    else:
        st = himuon_ns_tiled_hw(n, *ptrs, T, Tw, K, a, b, c, code, compute, *ws)
    if st != OK:
        raise HimuonError(st, "himuon_ns_tiled" if Tw is None or Tw == T else "himuon_ns_tiled_hw")
    _keep_alive(fresh, stream, dev)
    return outputs


def ns_gemm(inputs, outputs=None, T=0, K=5, coeffs=QUINTIC, compute=COMPUTE_DEFAULT,
            chunk_budget_bytes=0, workspace=None, stream=None, Tw=None):
    """Phi_K of every whole matrix (T = 0) or Phi_{K,T} with T x T tiles
    (T >= 1, e.g. 512) through library GEMMs, in one call; with ``Tw`` the
    tiles are T x Tw (rows x columns). Arguments and return value as
    ``ns_tiled``; ``workspace`` (if given) must hold
    ``himuon_ns_gemm_hw_workspace_size`` bytes for these shapes."""
    import torch
    inputs = list(inputs)
    if not inputs:
        raise ValueError("no matrices")
    code = _dtype_code(inputs[0])
    dev = inputs[0].device
    for x in inputs:
        if x.dim() != 2 or not x.is_cuda or x.device != dev or _dtype_code(x) != code or x.stride(1) != 1:
            raise ValueError("inputs must be 2-D row-major CUDA tensors of one dtype on one device")
    fresh = []  # tensors allocated here for the call
    if outputs is None:
        outputs = [torch.empty_like(x, memory_format=torch.contiguous_format) for x in inputs]
        fresh += outputs
    outputs = list(outputs)
    if len(outputs) != len(inputs):
        raise ValueError("inputs and outputs differ in length")
    for x, y in zip(inputs, outputs):
        if y.shape != x.shape or y.dtype != x.dtype or y.device != dev or y.stride(1) != 1:
            raise ValueError("each output must match its input's shape, dtype and device")
    n = len(inputs)
    a, b, c = coeffs
    rows = [x.shape[0] for x in inputs]
    cols = [x.shape[1] for x in inputs]
    Th, Tw = int(T), int(T if Tw is None else Tw)
    need = himuon_ns_gemm_hw_workspace_size(rows, cols, Th, Tw, code, compute, K, a, b, c, chunk_budget_bytes)
    if need == 0:
        raise HimuonError(ERR_INVALID_ARG, "himuon_ns_gemm_hw_workspace_size")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
        fresh.append(workspace)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    st = himuon_ns_gemm_hw(
        n, [x.data_ptr() for x in inputs], [y.data_ptr() for y in outputs], rows, cols,
        [x.stride(0) for x in inputs], [y.stride(0) for y in outputs],
        Th, Tw, K, a, b, c, code, compute, workspace.data_ptr(), workspace.numel() * workspace.element_size(),
        chunk_budget_bytes, stream.cuda_stream)
    if st != OK:
        raise HimuonError(st, "himuon_ns_gemm_hw")
    _keep_alive(fresh, stream, dev)
    return outputs


def step(weights, grads, moms, T=512, K=5, coeffs=QUINTIC, lr=0.02, momentum=0.95, weight_decay=0.0,
         nesterov=True, scale_c=0.2, compute=COMPUTE_DEFAULT, chunk_budget_bytes=0, workspace=None, stream=None):
    """One HiMuon optimizer step (Alg. 1) on every matrix, in one library
    call: ``weights`` and ``moms`` are updated in place from ``grads``. All
    three are lists of 2-D CUDA tensors of one dtype, matrix l sharing one
    shape and row stride across the three lists. T = 0 is the full-matrix
    branch. Returns ``weights``."""
    import torch
    weights, grads, moms = list(weights), list(grads), list(moms)
    if not weights or len(grads) != len(weights) or len(moms) != len(weights):
        raise ValueError("weights, grads and moms must be equally long, non-empty lists")
    code = _dtype_code(weights[0])
    dev = weights[0].device
    for w, g, m in zip(weights, grads, moms):
        for x in (w, g, m):
            if x.dim() != 2 or not x.is_cuda or x.device != dev or _dtype_code(x) != code or x.stride(1) != 1:
                raise ValueError("matrices must be 2-D row-major CUDA tensors of one dtype on one device")
        if g.shape != w.shape or m.shape != w.shape or g.stride(0) != w.stride(0) or m.stride(0) != w.stride(0):
            raise ValueError("W, G and M of a matrix must share shape and row stride")
    a, b, c = coeffs
    rows = [w.shape[0] for w in weights]
    cols = [w.shape[1] for w in weights]
    need = himuon_step_workspace_size(rows, cols, T, code, compute, K, a, b, c, chunk_budget_bytes)
    if need == 0:
        raise HimuonError(ERR_INVALID_ARG, "himuon_step_workspace_size")
    fresh = []
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
        fresh.append(workspace)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    st = himuon_step(
        len(weights), [w.data_ptr() for w in weights], [g.data_ptr() for g in grads], [m.data_ptr() for m in moms],
        rows, cols, [w.stride(0) for w in weights], T, K, a, b, c, lr, momentum, weight_decay, nesterov, scale_c,
        code, compute, workspace.data_ptr(), workspace.numel() * workspace.element_size(), chunk_budget_bytes,
        stream.cuda_stream)
    if st != OK:
        raise HimuonError(st, "himuon_step")
    _keep_alive(fresh, stream, dev)
    return weights


class HiMuon:
    """Optimizer state around ``himuon_step`` (Alg. 1): one momentum buffer per
    matrix (zero at the start, independent of T) and a device workspace
    cached across steps. ``reconfigure(T)`` changes the tile size at run time
    (Sec. 4.4.3) and keeps the momentum; T = 0 is the full-matrix branch.
    Every step is one library call over all matrices (cross-layer batching,
    Sec. 4.4.2). With ``tune`` (default), a tile size served by the library
    GEMMs has its GEMM kernels chosen by timing at (re)configuration. With
    ``capture``, the step is recorded once into a plan (a HIP graph, rebuilt
    by ``reconfigure`` and when the gradient buffers change) and each step is
    one graph launch."""

    def __init__(self, params, T=512, K=5, coeffs=QUINTIC, lr=0.02, momentum=0.95, weight_decay=0.0,
                 nesterov=True, scale_c=0.2, compute=COMPUTE_DEFAULT, chunk_budget_bytes=0, tune=True,
                 capture=False):
        import torch
        self.params = list(params)
        if not self.params:
            raise ValueError("no parameters")
        self.moms = [torch.zeros_like(p, memory_format=torch.contiguous_format) for p in self.params]
        for p, m in zip(self.params, self.moms):
            if p.dim() != 2 or p.stride(1) != 1 or p.stride(0) != m.stride(0):
                raise ValueError("parameters must be contiguous 2-D matrices")
        self.K, self.coeffs, self.lr, self.momentum = K, coeffs, lr, momentum
        self.weight_decay, self.nesterov, self.scale_c = weight_decay, nesterov, scale_c
        self.compute, self.chunk_budget_bytes = compute, chunk_budget_bytes
        self.tune = tune
        self.capture = capture
        self._workspace = None
        self._streams = set()
        self._plan = None
        self._plan_key = None
        self.reconfigure(T)

    def reconfigure(self, T):
        """Set the tile size for the following steps; the plan's workspace is
        sized once here and reused by every step."""
        import torch
        a, b, c = self.coeffs
        code = _dtype_code(self.params[0])
        need = himuon_step_workspace_size([p.shape[0] for p in self.params], [p.shape[1] for p in self.params],
                                          T, code, self.compute, self.K, a, b, c, self.chunk_budget_bytes)
        if need == 0:
            raise HimuonError(ERR_INVALID_ARG, "himuon_step_workspace_size")
        if self._workspace is None or self._workspace.numel() < need:
            if self._workspace is not None:
                # steps enqueued on other streams may still use the old workspace
                torch.cuda.synchronize(self._workspace.device)
            self._workspace = torch.empty(need, dtype=torch.uint8, device=self.params[0].device)
            self._streams = set()  # streams the new workspace has been marked as used on
        if self.tune and T not in (32, 64, 128, 256):
            gemm_tune([tuple(p.shape) for p in self.params], T, code, K=self.K, coeffs=self.coeffs,
                      compute=self.compute, chunk_budget_bytes=self.chunk_budget_bytes, workspace=self._workspace)
        self.T = T
        if self._plan is not None:  # the recorded step belongs to the previous tile size
            self._plan.close()
            self._plan = None

    def _step_plan(self, grads):
        """The recorded step for these gradient buffers (re-recorded when they change)."""
        import torch
        key = tuple(g.data_ptr() for g in grads)
        if self._plan is None or self._plan_key != key:
            if self._plan is not None:
                self._plan.close()
            a, b, c = self.coeffs
            code = _dtype_code(self.params[0])
            with torch.cuda.device(self.params[0].device):
                st, h = himuon_plan_step(
                    len(self.params), [p.data_ptr() for p in self.params], [g.data_ptr() for g in grads],
                    [m.data_ptr() for m in self.moms], [p.shape[0] for p in self.params],
                    [p.shape[1] for p in self.params], [p.stride(0) for p in self.params], self.T, self.K, a, b, c,
                    self.lr, self.momentum, self.weight_decay, self.nesterov, self.scale_c, code, self.compute,
                    self._workspace.data_ptr(), self._workspace.numel(), self.chunk_budget_bytes)
            if st != OK:
                raise HimuonError(st, "himuon_plan_step")
            self._plan = Plan(h, (list(grads),))
            self._plan_key = key
        return self._plan

    def step(self, grads, stream=None):
        if self.capture:
            # one graph launch per step: the gradient buffers must keep their storage between steps
            for g, p in zip(grads, self.params):
                if g.shape != p.shape or g.dtype != p.dtype or g.stride(0) != p.stride(0):
                    raise ValueError("each gradient must match its parameter's shape, dtype and row stride")
            self._step_plan(list(grads)).launch(stream)
        else:
            step(self.params, grads, self.moms, T=self.T, K=self.K, coeffs=self.coeffs, lr=self.lr,
                 momentum=self.momentum, weight_decay=self.weight_decay, nesterov=self.nesterov,
                 scale_c=self.scale_c, compute=self.compute, chunk_budget_bytes=self.chunk_budget_bytes,
                 workspace=self._workspace, stream=stream)
        if stream is not None and stream not in self._streams:
            # the cached workspace (and the momenta) are in use on `stream` too;
            # the allocator keeps the record for the life of each block, so
            # once per stream and workspace is enough
            _keep_alive([self._workspace] + self.moms, stream, self._workspace.device)
            self._streams.add(stream)
        return self.params
