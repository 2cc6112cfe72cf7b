"""himuon_ns_tiled_noalloc (the entry point that allocates nothing) against
himuon_ns_tiled, through the C ABI.

Both run the same tile kernels, so the outputs must be equal bit for bit.
Two calls in a row share the library's device-side descriptor table; the
second is smaller, so entries the first call left behind beyond its matrix
count must not matter. A call with the most matrices the table holds goes
through more than one upload launch.
"""
import numpy as np
import pytest
import torch

import paper_2606_27216_amd as hm
import workloads
from parity import COEF32

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _args(mats, outs):
    return dict(n_mats=len(mats), in_ptrs=[x.data_ptr() for x in mats], out_ptrs=[y.data_ptr() for y in outs],
                rows=[x.shape[0] for x in mats], cols=[x.shape[1] for x in mats],
                ld_in=[x.stride(0) for x in mats], ld_out=[y.stride(0) for y in outs])


def noalloc(mats, T, K=5, budget=0, dtype=hm.BF16, compute=hm.COMPUTE_DEFAULT):
    outs = [torch.empty_like(x) for x in mats]
    torch.cuda.synchronize()
    st = hm.himuon_ns_tiled_noalloc(**_args(mats, outs), T=T, K=K, a=COEF32[0], b=COEF32[1], c=COEF32[2],
                                    dtype=dtype, compute=compute, chunk_budget_bytes=budget,
                                    stream=torch.cuda.current_stream().cuda_stream)
    assert st == hm.OK, hm.himuon_status_string(st)
    torch.cuda.synchronize()
    return outs


def reference(mats, T, K=5, budget=0, compute=hm.COMPUTE_DEFAULT):
    outs = hm.ns_tiled(mats, T=T, K=K, coeffs=COEF32, compute=compute, chunk_budget_bytes=budget)
    torch.cuda.synchronize()
    return outs


@pytest.mark.parametrize("dtype,T", [("bf16", 128), ("bf16", 32), ("bf16", 256), ("f32", 64)])
def test_noalloc_equals_workspace_entry_point_twice(dtype, T):
    code = hm.BF16 if dtype == "bf16" else hm.F32
    first = [workloads.student_t(h, w, 300 + i, dtype, DEV)
             for i, (h, w) in enumerate([(3 * T + 5, 2 * T), (T, 5 * T + 3), (700, 33), (1, 1), (257, 300)])]
    second = [workloads.student_t(h, w, 310 + i, dtype, DEV) for i, (h, w) in enumerate([(2 * T, T + 9)])]
    for name, mats, budget in (("first", first, 3 * 2 * T * T * (2 if dtype == "bf16" else 4)), ("second", second, 0)):
        announce(f"noalloc {dtype} T={T}, {name} call: {len(mats)} matrices, budget {budget}")
        got = noalloc(mats, T, budget=budget, dtype=code)
        ref = reference(mats, T, budget=budget)
        for a, b in zip(got, ref):
            assert torch.equal(a, b)


def test_noalloc_most_matrices_then_fewer():
    """HIMUON_NOALLOC_MAX_MATS matrices (22 upload launches of 48
    descriptors), then 3 matrices: each equal to the workspace entry point."""
    n = hm.NOALLOC_MAX_MATS
    announce(f"noalloc bf16 T=64 with {n} matrices, then 3")
    big = workloads.gaussian(n, 96, 320, "bf16", DEV)
    mats = [big[i:i + 1] for i in range(n)]  # 1 x 96 rows of one buffer, each its own matrix
    outs = noalloc(mats, 64)
    ref = reference(mats, 64)
    for a, b in zip(outs, ref):
        assert torch.equal(a, b)
    small = [workloads.gaussian(130, 70, 321 + i, "bf16", DEV) for i in range(3)]
    for a, b in zip(noalloc(small, 64), reference(small, 64)):
        assert torch.equal(a, b)


def test_noalloc_rejects_what_it_cannot_serve():
    x = workloads.gaussian(300, 300, 330, "f32", DEV)
    y = torch.zeros_like(x)
    kw = dict(**_args([x], [y]), K=5, a=COEF32[0], b=COEF32[1], c=COEF32[2], chunk_budget_bytes=0,
              stream=torch.cuda.current_stream().cuda_stream)
    # fp32 256-tiles run on the library-GEMM route, which needs a workspace
    assert hm.himuon_ns_tiled_noalloc(T=256, dtype=hm.F32, compute=hm.COMPUTE_DEFAULT, **kw) == hm.ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert not torch.any(y)
