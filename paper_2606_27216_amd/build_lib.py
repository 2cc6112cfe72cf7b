"""Build libhimuon.so (gfx950) in-tree with hipcc.

    python -m paper_2606_27216_amd.build_lib

The library holds the HIP kernel family and the C ABI declared in
include/himuon.h. Every HIP source is compiled with packed-fp32 VALU ops
disabled (``-packed-fp32-ops``); the host pass prints a harmless warning
that it does not know that feature.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIBRARY = os.path.join(PKG, "libhimuon.so")
BUILD_DIR = os.path.join(PKG, "_build")
ARCH = "gfx950"

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"),
]
# (source, extra flags). The fp16 kernel keeps its MFMA accumulators in
# architectural VGPRs, where the vector ALU converts them after each product;
# the fp32/bf16 kernels keep the compiler's default register classes.
SOURCES = [
    ("ns_tiled_kernels.hip", []),
    ("ns_tiled_f16.hip", ["-mllvm", "-amdgpu-mfma-vgpr-form"]),
    ("ns_tiled_noalloc.hip", []),
    ("ns_rect.hip", []),
    ("ns_gemm_kernels.hip", []),
    ("optim_kernels.hip", []),
    ("himuon_api.cpp", []),
    ("ns_gemm_path.cpp", []),
    ("himuon_step.cpp", []),
    ("himuon_plan.cpp", []),
    ("calib_mfma.hip", []),
]
# The whole-matrix and large-tile path runs its Newton-Schulz GEMMs on hipBLASLt.
LINK_LIBS = ["-lhipblaslt"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{msgs}")
    if msgs.strip() and verbose:
        print(msgs)


def build(verbose: bool = False, jobs: int = 0) -> str:
    """Compile every source (in parallel, `jobs` at a time; 0: up to 8) and
    link the library."""
    from concurrent.futures import ThreadPoolExecutor

    os.makedirs(BUILD_DIR, exist_ok=True)
    cmds, objs = [], []
    for src, extra in SOURCES:
        obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
        cmds.append([hipcc()] + COMMON + extra + ["-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    jobs = jobs or min(8, len(cmds), os.cpu_count() or 1)
    with ThreadPoolExecutor(max_workers=jobs) as pool:
        for f in [pool.submit(_run, c, verbose) for c in cmds]:
            f.result()
    tmp = LIBRARY + ".tmp"
    _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC"] + objs + LINK_LIBS + ["-o", tmp], verbose)
    os.replace(tmp, LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
