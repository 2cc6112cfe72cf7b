"""fp64 CPU oracle for the tiled Newton–Schulz map (test infrastructure).

TEST INFRASTRUCTURE ONLY: imported by tests/, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py``. The product path (the HIP library and
its Python binding) never imports this package, and this package imports
nothing from the product path.

The arithmetic lives in ``himuon_oracle.c`` (plain fp64 loops, OpenMP over
tiles); this module only compiles it with gcc and marshals numpy arrays.

Functions (all inputs are converted to float64 exactly; coefficients are
taken as given, so callers that want the GPU's fp32 coefficients pass
``float(np.float32(x))``):

* ``phi_k(A, K, a, b, c)``          Φ_K(A), Sec. 2.2 incl. orientation rule.
* ``ns_tiled(A, T, K, a, b, c)``    Φ_{K,T}(A), eq. (tiled_ns).
* ``ns_tiled_hw(A, Th, Tw, K, a, b, c)``  the same map with Th×Tw tiles (the
                                    tile-shape study's rectangular tiles).
* ``ns_tiles(A, T, K, a, b, c, ids)`` selected tiles of Φ_{K,T}, each T×T.
* ``tile_count(H, W, T)``           R·C of the tiling operator B_T.
* ``himuon_step(W, M, G, T, K, a, b, c, lr, beta, wd, nesterov, scale_c)``
                                    one optimizer step of Alg. 1 (T = 0: the
                                    full-matrix branch); returns (W', M', U).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "himuon_oracle.c")
LIBRARY = os.path.join(_HERE, "libhimuon_oracle.so")

_lib = None
_lib_path = None


def build(source: str = SOURCE, output: str = LIBRARY, openmp: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no -march, so no FMA contraction)."""
    cmd = ["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-Wall", "-Wextra"]
    if openmp:
        cmd.append("-fopenmp")
    cmd += [source, "-o", output + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(output + ".tmp", output)
    return output


def _bind(lib):
    d = ctypes.c_double
    i64 = ctypes.c_int64
    p = ctypes.c_void_p
    lib.oracle_phi_k.argtypes = [p, i64, i64, i64, ctypes.c_int, d, d, d, p, i64]
    lib.oracle_phi_k.restype = ctypes.c_int
    lib.oracle_tile_count.argtypes = [i64, i64, i64]
    lib.oracle_tile_count.restype = i64
    lib.oracle_ns_tile.argtypes = [p, i64, i64, i64, i64, i64, ctypes.c_int, d, d, d, p]
    lib.oracle_ns_tile.restype = ctypes.c_int
    lib.oracle_ns_tiled.argtypes = [p, i64, i64, i64, i64, ctypes.c_int, d, d, d, p, i64]
    lib.oracle_ns_tiled.restype = ctypes.c_int
    lib.oracle_ns_tiled_hw.argtypes = [p, i64, i64, i64, i64, i64, ctypes.c_int, d, d, d, p, i64]
    lib.oracle_ns_tiled_hw.restype = ctypes.c_int
    lib.oracle_ns_tiles.argtypes = [p, i64, i64, i64, i64, ctypes.c_int, d, d, d, i64, p, p]
    lib.oracle_ns_tiles.restype = ctypes.c_int
    lib.oracle_himuon_step.argtypes = [p, p, p, i64, i64, i64, ctypes.c_int, d, d, d, d, d, d, ctypes.c_int,
                                       d, p]
    lib.oracle_himuon_step.restype = ctypes.c_int
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    return lib


def load(path: str | None = None):
    """Load (building first if absent) the oracle library; ``path`` selects
    another build of the same source, e.g. a deliberately mutated copy."""
    global _lib, _lib_path
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIBRARY) or os.path.getmtime(LIBRARY) < os.path.getmtime(SOURCE):
            build()
        _lib = _bind(ctypes.CDLL(LIBRARY))
        _lib_path = LIBRARY
    return _lib


def _f64(A):
    A = np.asarray(A, dtype=np.float64)
    if A.ndim != 2:
        raise ValueError("expected a 2-D matrix")
    return np.ascontiguousarray(A)


def _check(st, what):
    if st != 0:
        raise RuntimeError(f"oracle {what} failed with status {st}")


def phi_k(A, K, a, b, c, lib=None):
    lib = lib or load()
    A = _f64(A)
    H, W = A.shape
    Y = np.empty_like(A)
    _check(lib.oracle_phi_k(A.ctypes.data, H, W, W, int(K), float(a), float(b), float(c),
                            Y.ctypes.data, W), "phi_k")
    return Y


def ns_tiled(A, T, K, a, b, c, lib=None):
    lib = lib or load()
    A = _f64(A)
    H, W = A.shape
    Y = np.empty_like(A)
    _check(lib.oracle_ns_tiled(A.ctypes.data, H, W, W, int(T), int(K), float(a), float(b), float(c),
                               Y.ctypes.data, W), "ns_tiled")
    return Y


def ns_tiled_hw(A, Th, Tw, K, a, b, c, lib=None):
    lib = lib or load()
    A = _f64(A)
    H, W = A.shape
    Y = np.empty_like(A)
    _check(lib.oracle_ns_tiled_hw(A.ctypes.data, H, W, W, int(Th), int(Tw), int(K), float(a), float(b), float(c),
                                  Y.ctypes.data, W), "ns_tiled_hw")
    return Y


def ns_tiles(A, T, K, a, b, c, tile_ids, lib=None):
    lib = lib or load()
    A = _f64(A)
    H, W = A.shape
    ids = np.ascontiguousarray(np.asarray(tile_ids, dtype=np.int64))
    Y = np.empty((len(ids), int(T), int(T)), dtype=np.float64)
    _check(lib.oracle_ns_tiles(A.ctypes.data, H, W, W, int(T), int(K), float(a), float(b), float(c),
                               len(ids), ids.ctypes.data, Y.ctypes.data), "ns_tiles")
    return Y


def tile_count(H, W, T, lib=None):
    lib = lib or load()
    return int(lib.oracle_tile_count(int(H), int(W), int(T)))


def himuon_step(W, M, G, T, K, a, b, c, lr, beta, weight_decay, nesterov, scale_c, lib=None):
    """Alg. 1 for one matrix: returns new copies (W', M', U); inputs untouched."""
    lib = lib or load()
    W1 = _f64(W).copy()
    M1 = _f64(M).copy()
    G = _f64(G)
    if W1.shape != M1.shape or W1.shape != G.shape:
        raise ValueError("W, M and G must have one shape")
    H, Wd = W1.shape
    U = np.empty_like(W1)
    _check(lib.oracle_himuon_step(W1.ctypes.data, M1.ctypes.data, G.ctypes.data, H, Wd, int(T), int(K),
                                  float(a), float(b), float(c), float(lr), float(beta), float(weight_decay),
                                  int(bool(nesterov)), float(scale_c), U.ctypes.data), "himuon_step")
    return W1, M1, U


def set_num_threads(n: int, lib=None) -> None:
    """Thread count of the oracle's OpenMP loops over tiles (through the
    OpenMP runtime the library is linked with; results do not depend on it,
    each tile being computed by one thread)."""
    lib = lib or load()
    f = lib.omp_set_num_threads
    f.argtypes = [ctypes.c_int]
    f.restype = None
    f(int(n))


def num_threads(lib=None):
    lib = lib or load()
    return int(lib.oracle_num_threads())
