"""Resource usage of every HIP kernel, as hipcc reports it for gfx950.

CPU-only: hipcc cross-compiles. The checks guard properties the kernels' speed
rests on. Nothing spills to scratch. No private variable is promoted into LDS
beside the kernels' own arrays: a struct with bool members once was, which
cost an LDS round trip and a full LDS wait per tile. The fused tile kernels
keep the occupancy that their persistent grid is sized for.
"""
import functools
import os
import re
import subprocess

import pytest

from paper_2606_27216_amd import build_lib as B

HIP_SOURCES = [(src, extra) for src, extra in B.SOURCES if src.endswith(".hip")]
LDS_PER_CU = 160 * 1024

# LDS bytes per workgroup of the fused bf16-storage kernels (map variants,
# c > 0): exactly the kernels' own arrays (Z copy, H/P blocks, reductions).
F16_LDS = {32: 8192, 64: 65536, 128: 77872, 256: 147552}
# tiles (workgroups) per CU that the grid sizing relies on
F16_WG_PER_CU = {32: 5, 64: 2, 128: 2, 256: 1}


def _hipcc_available():
    h = B.hipcc()
    return os.path.isabs(h) and os.path.exists(h)


pytestmark = pytest.mark.skipif(not _hipcc_available(), reason="hipcc not found")


@functools.lru_cache(maxsize=None)
def _resource_usage(src, extra):
    """{kernel symbol: {remark name: value}} from -Rpass-analysis=kernel-resource-usage."""
    cmd = ([B.hipcc()] + B.COMMON + list(extra) +
           ["--cuda-device-only", "-c", os.path.join(B.CSRC, src), "-o", os.devnull,
            "-Rpass-analysis=kernel-resource-usage"])
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-3000:]
    kernels, cur = {}, None
    for line in res.stderr.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", line)
        if m:
            cur = kernels.setdefault(m.group(1), {})
            continue
        m = re.search(r"remark:\s+([A-Za-z ]+?)(?: \[[^\]]*\])?: (\d+) \[-Rpass", line)
        if m and cur is not None:
            cur[m.group(1).strip()] = int(m.group(2))
    return kernels


def resource_usage(src, extra):
    return _resource_usage(src, tuple(extra))


@pytest.mark.parametrize("src,extra", HIP_SOURCES, ids=[s for s, _ in HIP_SOURCES])
def test_no_scratch_and_lds_within_a_cu(src, extra):
    kernels = resource_usage(src, extra)
    assert kernels, f"no kernels reported for {src}"
    for name, r in kernels.items():
        # no spill or private array in memory (spills into AGPRs or VGPR lanes
        # stay in registers and are allowed)
        assert r.get("ScratchSize") == 0, f"{name}: scratch {r.get('ScratchSize')} B/lane"
        assert r.get("LDS Size", 0) <= LDS_PER_CU, f"{name}: LDS {r.get('LDS Size')}"
        assert r.get("VGPRs", 0) + r.get("AGPRs", 0) <= 512, f"{name}: registers {r}"


def test_fused_tile_kernels_lds_and_occupancy():
    src, extra = next((s, e) for s, e in HIP_SOURCES if s == "ns_tiled_f16.hip")
    kernels = resource_usage(src, extra)
    seen = set()
    for name, r in kernels.items():
        m = re.search(r"ns_tiled_f16_kernelILi(\d+)ELi\d+ELi0ELb0E", name)  # map kernel, c > 0
        if not m:
            continue
        T = int(m.group(1))
        seen.add(T)
        assert r["LDS Size"] == F16_LDS[T], f"T={T}: LDS {r['LDS Size']} B per workgroup, expected {F16_LDS[T]}"
        assert F16_WG_PER_CU[T] * r["LDS Size"] <= LDS_PER_CU
        waves_per_wg = {32: 4, 64: 4, 128: 2, 256: 4}[T]
        # workgroups per CU allowed by the waves per SIMD the registers leave
        assert r["Occupancy"] * 4 // waves_per_wg >= F16_WG_PER_CU[T], f"T={T}: occupancy {r['Occupancy']}"
    assert seen == set(F16_LDS), seen
