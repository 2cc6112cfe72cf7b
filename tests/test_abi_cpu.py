"""The C ABI on a machine without a GPU: exports, validation, planner."""
import ctypes
import json
import os
import re

import pytest

import paper_2606_27216_amd as hm
import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLD = json.load(open(os.path.join(ROOT, "tests", "golden", "paper_constants.json")))
FAKE = 0x10000  # a non-null pointer value; validation fails before it is used


def declared_functions():
    src = open(os.path.join(ROOT, "include", "himuon.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(himuon_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 7
    lib = ctypes.CDLL(hm.LIBRARY)
    for n in names:
        assert hasattr(lib, n), f"{n} is declared in himuon.h but not exported"


def test_version_and_strings():
    assert hm.himuon_version() >= 100
    for st in (hm.OK, hm.ERR_INVALID_ARG, hm.ERR_UNSUPPORTED, hm.ERR_WORKSPACE, hm.ERR_HIP, hm.ERR_RANGE):
        assert hm.himuon_status_string(st) != "unknown status"
    assert hm.himuon_status_string(12345) == "unknown status"


def test_workspace_size():
    assert hm.himuon_ns_tiled_workspace_size(0) == 0
    assert hm.himuon_ns_tiled_workspace_size(1) == 256
    assert hm.himuon_ns_tiled_workspace_size(224) == 224 * 64


def test_call_workspace_size():
    """A call served by a fused kernel needs the descriptor table only; a
    256-tile call without a fused kernel (fp32 storage, bf16 operands) needs
    the library-GEMM path's workspace for T = 256."""
    a, b, c = hm.QUINTIC
    rows, cols = [1024, 2048, 300], [4096, 2048, 500]
    call = lambda T, dtype, compute=hm.COMPUTE_DEFAULT, budget=0, K=5: hm.himuon_ns_tiled_call_workspace_size(
        rows, cols, T, dtype, compute, K, a, b, c, budget)
    gemm = lambda T, dtype, compute=hm.COMPUTE_DEFAULT, budget=0: hm.himuon_ns_gemm_workspace_size(
        rows, cols, T, dtype, compute, 5, a, b, c, budget)
    for T in (32, 64, 128):
        for dtype in (hm.F32, hm.BF16):
            assert call(T, dtype) == hm.himuon_ns_tiled_workspace_size(3)
        assert call(T, hm.BF16, hm.COMPUTE_BF16) == hm.himuon_ns_tiled_workspace_size(3)
    assert call(256, hm.BF16) == hm.himuon_ns_tiled_workspace_size(3)  # fused fp16-operand kernel
    assert call(256, hm.F32) == gemm(256, hm.F32) > (64 << 20)
    assert call(256, hm.BF16, hm.COMPUTE_BF16) == gemm(256, hm.BF16, hm.COMPUTE_BF16)
    budget = 4 * (2 * 256 * 256 + 2 * 256 * 256) * 4  # four fp32 256-problems per chunk
    assert call(256, hm.F32, budget=budget) == gemm(256, hm.F32, budget=budget) < call(256, hm.F32)
    # rejected calls: no size
    assert call(48, hm.BF16) == 0 and call(512, hm.BF16) == 0
    assert call(128, hm.F32, hm.COMPUTE_F16) == 0
    assert hm.himuon_ns_tiled_call_workspace_size(rows, cols, 128, hm.BF16, hm.COMPUTE_DEFAULT, 5, 50.0, 0.0, 0.0) == 0


def _call(**kw):
    args = dict(n_mats=1, in_ptrs=[FAKE], out_ptrs=[FAKE], rows=[64], cols=[64], ld_in=None, ld_out=None,
                T=32, K=5, a=3.4445, b=-4.775, c=2.0315, dtype=hm.BF16, compute=hm.COMPUTE_DEFAULT,
                workspace=FAKE, workspace_bytes=256, chunk_budget_bytes=0, stream=None)
    args.update(kw)
    return hm.himuon_ns_tiled(**args)


@pytest.mark.parametrize("kw,status", [
    (dict(in_ptrs=[0]), hm.ERR_INVALID_ARG),
    (dict(out_ptrs=[0]), hm.ERR_INVALID_ARG),
    (dict(rows=[0]), hm.ERR_INVALID_ARG),
    (dict(cols=[-3]), hm.ERR_INVALID_ARG),
    (dict(ld_in=[63]), hm.ERR_INVALID_ARG),
    (dict(ld_out=[10]), hm.ERR_INVALID_ARG),
    (dict(K=-1), hm.ERR_INVALID_ARG),
    (dict(a=float("nan")), hm.ERR_INVALID_ARG),
    (dict(c=float("inf")), hm.ERR_INVALID_ARG),
    (dict(dtype=7), hm.ERR_INVALID_ARG),
    (dict(compute=9), hm.ERR_INVALID_ARG),
    (dict(T=48), hm.ERR_UNSUPPORTED),
    (dict(T=512), hm.ERR_UNSUPPORTED),
    (dict(dtype=hm.F32, compute=hm.COMPUTE_F16), hm.ERR_UNSUPPORTED),
    (dict(dtype=hm.BF16, compute=hm.COMPUTE_F32), hm.ERR_UNSUPPORTED),
    (dict(workspace=0), hm.ERR_WORKSPACE),
    (dict(workspace_bytes=255), hm.ERR_WORKSPACE),
    (dict(chunk_budget_bytes=100), hm.ERR_WORKSPACE),
    (dict(compute=hm.COMPUTE_F16, a=50.0, b=0.0, c=0.0), hm.ERR_RANGE),
    # DEFAULT never falls back to bf16 operands on its own
    (dict(a=50.0, b=0.0, c=0.0), hm.ERR_RANGE),
    # 256-tiles without a fused kernel run on the GEMM path, whose workspace is larger
    (dict(T=256, dtype=hm.F32), hm.ERR_WORKSPACE),
    (dict(T=256, compute=hm.COMPUTE_BF16), hm.ERR_WORKSPACE),
    # 2^32 tiles in one call (the kernels number tiles with 32-bit ids)
    (dict(rows=[1 << 37], cols=[32]), hm.ERR_UNSUPPORTED),
])
def test_validation_rejects_before_any_hip_call(kw, status):
    assert _call(**kw) == status


def test_noalloc_validation_rejects_before_any_hip_call():
    """The entry point that allocates nothing validates as himuon_ns_tiled,
    and rejects more matrices than its device table holds."""
    kw = dict(n_mats=1, in_ptrs=[FAKE], out_ptrs=[FAKE], rows=[64], cols=[64], ld_in=None, ld_out=None, T=32, K=5,
              a=3.4445, b=-4.775, c=2.0315, dtype=hm.BF16, compute=hm.COMPUTE_DEFAULT, chunk_budget_bytes=0,
              stream=None)
    for over, status in ((dict(rows=[0]), hm.ERR_INVALID_ARG), (dict(T=48), hm.ERR_UNSUPPORTED),
                         (dict(a=50.0, b=0.0, c=0.0), hm.ERR_RANGE), (dict(chunk_budget_bytes=100), hm.ERR_WORKSPACE),
                         (dict(T=256, dtype=hm.F32), hm.ERR_UNSUPPORTED)):
        assert hm.himuon_ns_tiled_noalloc(**{**kw, **over}) == status, over
    n = hm.NOALLOC_MAX_MATS + 1
    assert hm.himuon_ns_tiled_noalloc(**{**kw, "n_mats": n, "in_ptrs": [FAKE] * n, "out_ptrs": [FAKE] * n,
                                         "rows": [64] * n, "cols": [64] * n}) == hm.ERR_WORKSPACE


def test_plan_null_handles():
    assert hm.himuon_plan_launch(None, None) == hm.ERR_INVALID_ARG
    hm.himuon_plan_destroy(None)  # a no-op


def test_null_arrays_rejected():
    L = hm.lib()
    assert L.himuon_ns_tiled(1, None, None, None, None, None, None, 32, 5, 1.0, 0.0, 0.0, 1, 0,
                             None, 0, 0, None) == hm.ERR_INVALID_ARG
    assert L.himuon_ns_tiled(0, None, None, None, None, None, None, 32, 5, 1.0, 0.0, 0.0, 1, 0,
                             None, 0, 0, None) == hm.ERR_INVALID_ARG


def test_select_compute():
    a, b, c = hm.QUINTIC
    assert hm.himuon_select_compute(hm.F32, hm.COMPUTE_DEFAULT, 5, a, b, c) == hm.COMPUTE_F32
    assert hm.himuon_select_compute(hm.BF16, hm.COMPUTE_DEFAULT, 5, a, b, c) == hm.COMPUTE_F16
    assert hm.himuon_select_compute(hm.BF16, hm.COMPUTE_DEFAULT, 8, a, b, c) == hm.COMPUTE_F16
    assert hm.himuon_select_compute(hm.BF16, hm.COMPUTE_BF16, 5, a, b, c) == hm.COMPUTE_BF16
    # iterates that grow without bound cannot use fp16 operands; DEFAULT
    # reports that instead of switching to bf16 operands on its own
    assert hm.himuon_select_compute(hm.BF16, hm.COMPUTE_DEFAULT, 20, 2.0, 0.0, 0.0) == hm.ERR_RANGE
    assert hm.himuon_select_compute(hm.BF16, hm.COMPUTE_F16, 20, 2.0, 0.0, 0.0) == hm.ERR_RANGE
    assert hm.himuon_select_compute(hm.BF16, hm.COMPUTE_BF16, 20, 2.0, 0.0, 0.0) == hm.COMPUTE_BF16
    assert hm.himuon_select_compute(hm.BF16, hm.COMPUTE_DEFAULT, 5, 4.0, -6.0, 3.0) == hm.ERR_RANGE
    # the textbook cubic iteration stays bounded
    assert hm.himuon_select_compute(hm.BF16, hm.COMPUTE_DEFAULT, 60, 1.5, -0.5, 0.0) == hm.COMPUTE_F16
    # one step's operator a I + P carries |a| itself: a large a alone must
    # move the call off fp16 operands
    assert hm.himuon_select_compute(hm.BF16, hm.COMPUTE_DEFAULT, 1, 20000.0, 0.0, 0.0) == hm.ERR_RANGE
    assert hm.himuon_select_compute(hm.BF16, hm.COMPUTE_F16, 1, 20000.0, 0.0, 0.0) == hm.ERR_RANGE


def _qwen(model):
    shapes = GOLD["qwen3_block_shapes"][model] * 28
    return [h for h, _ in shapes], [w for _, w in shapes]


def test_planner_reproduces_paper_chunking():
    """Sec. 6.4, T = 512: Qwen3-0.6B's 1680 tiles take one call, Qwen3-1.7B's
    5376 take two chunks of 2688 (the paper gives no
    budget; any budget between 2688 and 5375 one-MiB tiles gives this)."""
    ch = GOLD["cross_layer_chunking"]
    budget = 4 << 30  # 4 GiB; a T=512 bf16 tile stands for 2*512*512*2 B = 1 MiB
    total, bounds = hm.himuon_plan_chunks(*_qwen("0.6B"), ch["T"], hm.BF16, budget)
    assert total == ch["0.6B_total_tiles"]
    assert [bounds[i + 1] - bounds[i] for i in range(len(bounds) - 1)] == ch["0.6B_chunks"]
    total, bounds = hm.himuon_plan_chunks(*_qwen("1.7B"), ch["T"], hm.BF16, budget)
    assert total == ch["1.7B_total_tiles"]
    assert [bounds[i + 1] - bounds[i] for i in range(len(bounds) - 1)] == ch["1.7B_chunks"]


def test_planner_7b_stack_16gb():
    """32 layers of 7B shapes at T=128, bf16: 395,264 tiles; 25.9 GB of tile
    bytes against a 16 GB budget gives two chunks of 197,632."""
    import workloads
    shapes = workloads.stack_7b_shapes(32)
    rows, cols = [h for h, _ in shapes], [w for _, w in shapes]
    total, bounds = hm.himuon_plan_chunks(rows, cols, 128, hm.BF16, 16 * 10 ** 9)
    assert total == 395264 == sum(oracle.tile_count(h, w, 128) for h, w in shapes)
    assert bounds == [0, 197632, 395264]
    for T, n in ((32, 6324224), (64, 1581056), (256, 98816)):
        assert hm.himuon_plan_chunks(rows, cols, T, hm.BF16, 0)[0] == n


@pytest.mark.parametrize("budget_tiles", [1, 2, 3, 7, 100, 10 ** 6])
def test_planner_fewest_balanced_chunks(budget_tiles):
    rows, cols = [100, 257, 33, 1], [300, 129, 4096, 1]
    T = 32
    per_tile = 2 * T * T * 4
    total, bounds = hm.himuon_plan_chunks(rows, cols, T, hm.F32, budget_tiles * per_tile)
    assert total == sum(oracle.tile_count(h, w, T) for h, w in zip(rows, cols))
    sizes = [bounds[i + 1] - bounds[i] for i in range(len(bounds) - 1)]
    n = len(sizes)
    assert bounds[0] == 0 and bounds[-1] == total
    assert max(sizes) <= budget_tiles and max(sizes) - min(sizes) <= 1
    assert n == -(-total // min(budget_tiles, total))  # fewest that fit


def test_planner_errors():
    with pytest.raises(hm.HimuonError):
        hm.himuon_plan_chunks([10], [10], 32, hm.BF16, 1000)  # budget below one tile
    with pytest.raises(hm.HimuonError):
        hm.himuon_plan_chunks([0], [10], 32, hm.BF16, 0)


# ---- the library-GEMM path (himuon_ns_gemm): sizing and validation, no HIP call

def test_gemm_workspace_size():
    a, b, c = hm.QUINTIC
    ws = lambda rows, cols, T, dtype=hm.BF16, budget=0, compute=hm.COMPUTE_DEFAULT, K=5: \
        hm.himuon_ns_gemm_workspace_size(rows, cols, T, dtype, compute, K, a, b, c, budget)
    lt = 64 << 20
    # one 7B layer as whole matrices: the 4096 x 4096 group (4 problems of X, X', A, B in fp16) dominates
    layer_r, layer_c = [4096] * 4 + [11008, 11008, 4096], [4096] * 4 + [4096, 4096, 11008]
    assert ws(layer_r, layer_c, 0) >= 4 * 4 * 4096 * 4096 * 2 + lt
    # fp32 storage doubles the iterate bytes
    assert ws([512], [512], 0, hm.F32) - lt > ws([512], [512], 0) - lt
    # a chunk budget bounds the buffers; below one problem there is no plan
    one = 2 * (2 * 512 * 512 + 2 * 512 * 512)
    assert ws([4096], [4096], 512, budget=2 * one) < ws([4096], [4096], 512)
    assert ws([4096], [4096], 512, budget=one - 1) == 0
    assert ws([0], [64], 0) == 0
    assert ws([64], [64], -1) == 0
    assert ws([64], [64], 0, dtype=7) == 0
    assert ws([64], [64], 0, dtype=hm.F32, compute=hm.COMPUTE_F16) == 0
    assert ws([40000], [40000], 0) == 0  # Gram size above 32768
    # the fp16 iterate scale is capped (s^2 = min(m, 4096)), so any Gram size
    # up to the limit keeps fp16 operands by default; growing iterates cannot
    assert ws([20000], [20000], 0) >= 4 * 20000 * 20000 * 2
    assert ws([64], [64], 0, K=20) > 0
    assert hm.himuon_ns_gemm_workspace_size([64], [64], 0, hm.BF16, hm.COMPUTE_DEFAULT, 20, 2.0, 0.0, 0.0, 0) == 0
    assert hm.himuon_ns_gemm_workspace_size([64], [64], 0, hm.BF16, hm.COMPUTE_BF16, 20, 2.0, 0.0, 0.0, 0) > 0


def _gcall(**kw):
    args = dict(n_mats=1, in_ptrs=[FAKE], out_ptrs=[FAKE], rows=[64], cols=[64], ld_in=None, ld_out=None,
                T=0, K=5, a=3.4445, b=-4.775, c=2.0315, dtype=hm.BF16, compute=hm.COMPUTE_DEFAULT,
                workspace=FAKE, workspace_bytes=256, chunk_budget_bytes=0, stream=None)
    args.update(kw)
    return hm.himuon_ns_gemm(**args)


@pytest.mark.parametrize("kw,status", [
    (dict(in_ptrs=[0]), hm.ERR_INVALID_ARG),
    (dict(rows=[0]), hm.ERR_INVALID_ARG),
    (dict(ld_in=[63]), hm.ERR_INVALID_ARG),
    (dict(T=-1), hm.ERR_INVALID_ARG),
    (dict(K=-1), hm.ERR_INVALID_ARG),
    (dict(b=float("nan")), hm.ERR_INVALID_ARG),
    (dict(dtype=7), hm.ERR_INVALID_ARG),
    (dict(dtype=hm.F32, compute=hm.COMPUTE_BF16), hm.ERR_UNSUPPORTED),
    (dict(rows=[40000], cols=[40000]), hm.ERR_UNSUPPORTED),
    (dict(compute=hm.COMPUTE_F16, a=50.0, b=0.0, c=0.0), hm.ERR_RANGE),
    (dict(a=50.0, b=0.0, c=0.0), hm.ERR_RANGE),
    (dict(workspace=0), hm.ERR_WORKSPACE),
    (dict(workspace_bytes=1 << 20), hm.ERR_WORKSPACE),
    (dict(T=512, chunk_budget_bytes=100), hm.ERR_WORKSPACE),
])
def test_gemm_validation_rejects_before_any_hip_call(kw, status):
    assert _gcall(**kw) == status


# ---- the optimizer step (himuon_step): sizing and validation, no HIP call

def test_step_workspace_size():
    a, b, c = hm.QUINTIC
    ws = lambda rows, cols, T, dtype=hm.BF16, budget=0: \
        hm.himuon_step_workspace_size(rows, cols, T, dtype, hm.COMPUTE_DEFAULT, 5, a, b, c, budget)
    gemm = lambda rows, cols, T, dtype=hm.BF16, budget=0: \
        hm.himuon_ns_gemm_workspace_size(rows, cols, T, dtype, hm.COMPUTE_DEFAULT, 5, a, b, c, budget)
    # T = 512 and T = 0 run the library-GEMM path: the same plan as himuon_ns_gemm
    assert ws([1024] * 8, [1024] * 8, 512) == gemm([1024] * 8, [1024] * 8, 512)
    assert ws([300], [500], 0, hm.F32) == gemm([300], [500], 0, hm.F32)
    # T <= 128, bf16, fp16 operands, c > 0: the step runs inside the tile kernel; the workspace is
    # the two descriptor tables (64 + 16 bytes per matrix, each rounded up to 256)
    assert ws([1024] * 8, [1024] * 8, 128) == 512 + 256
    assert ws([1024] * 300, [1024] * 300, 64) == 19200 + 4864
    # T = 256 (no step variant of its kernel): the lookahead buffers of all matrices
    # plus two descriptor tables
    need = ws([1024] * 8, [1024] * 8, 256)
    assert need >= 8 * 1024 * 1024 * 2 and need < 8 * 1024 * 1024 * 2 + 4096
    assert ws([1024] * 8, [1024] * 8, 128, dtype=hm.F32) == 512 + 256  # fp32: inside the tile kernel too
    # a budget groups matrices; one matrix above it has no plan
    assert ws([1024] * 8, [1024] * 8, 256, budget=2 * 1024 * 1024 * 2) < need
    assert ws([1024] * 8, [1024] * 8, 256, budget=1024 * 1024 * 2 - 1) == 0
    assert ws([0], [64], 128) == 0
    assert ws([64], [64], -1) == 0


def _scall(**kw):
    args = dict(n_mats=1, weights=[FAKE], grads=[FAKE + 4096], moms=[FAKE + 8192], rows=[64], cols=[64], ld=None,
                T=128, K=5, a=3.4445, b=-4.775, c=2.0315, lr=0.02, momentum=0.95, weight_decay=0.0, nesterov=True,
                scale_c=0.2, dtype=hm.BF16, compute=hm.COMPUTE_DEFAULT, workspace=FAKE, workspace_bytes=256,
                chunk_budget_bytes=0, stream=None)
    args.update(kw)
    return hm.himuon_step(**args)


@pytest.mark.parametrize("kw,status", [
    (dict(weights=[0]), hm.ERR_INVALID_ARG),
    (dict(moms=[0]), hm.ERR_INVALID_ARG),
    (dict(grads=[FAKE]), hm.ERR_INVALID_ARG),       # G aliases W
    (dict(moms=[FAKE + 4096]), hm.ERR_INVALID_ARG),  # M aliases G
    (dict(rows=[0]), hm.ERR_INVALID_ARG),
    (dict(ld=[63]), hm.ERR_INVALID_ARG),
    (dict(T=-1), hm.ERR_INVALID_ARG),
    (dict(K=-1), hm.ERR_INVALID_ARG),
    (dict(lr=float("inf")), hm.ERR_INVALID_ARG),
    (dict(momentum=float("nan")), hm.ERR_INVALID_ARG),
    (dict(scale_c=float("nan")), hm.ERR_INVALID_ARG),
    (dict(dtype=7), hm.ERR_INVALID_ARG),
    (dict(T=0, dtype=hm.F32, compute=hm.COMPUTE_BF16), hm.ERR_UNSUPPORTED),
    (dict(T=0, compute=hm.COMPUTE_F16, a=50.0, b=0.0, c=0.0), hm.ERR_RANGE),
    (dict(workspace=0), hm.ERR_WORKSPACE),              # in-kernel route: no descriptor tables
    (dict(T=256, workspace_bytes=1024), hm.ERR_WORKSPACE),  # prologue/epilogue route: buffers do not fit
    (dict(T=512, workspace_bytes=1 << 20), hm.ERR_WORKSPACE),  # GEMM route
    (dict(chunk_budget_bytes=100), hm.ERR_WORKSPACE),
])
def test_step_validation_rejects_before_any_hip_call(kw, status):
    assert _scall(**kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(rows=[0]), hm.ERR_INVALID_ARG),
    (dict(T=-1), hm.ERR_INVALID_ARG),
    (dict(K=-1), hm.ERR_INVALID_ARG),
    (dict(dtype=7), hm.ERR_INVALID_ARG),
    (dict(dtype=hm.F32, compute=hm.COMPUTE_BF16), hm.ERR_UNSUPPORTED),
    (dict(workspace=0), hm.ERR_WORKSPACE),
    (dict(workspace_bytes=1024), hm.ERR_WORKSPACE),
])
def test_gemm_tune_validation_rejects_before_any_hip_call(kw, status):
    args = dict(rows=[64], cols=[64], T=0, dtype=hm.BF16, compute=hm.COMPUTE_DEFAULT, K=5, a=3.4445, b=-4.775,
                c=2.0315, workspace=FAKE, workspace_bytes=256, chunk_budget_bytes=0, stream=None)
    args.update(kw)
    assert hm.himuon_gemm_tune(**args) == status


def test_gemm_hw_workspace_and_validation():
    a, b, c = hm.QUINTIC
    ws = lambda rows, cols, Th, Tw, budget=0: \
        hm.himuon_ns_gemm_hw_workspace_size(rows, cols, Th, Tw, hm.BF16, hm.COMPUTE_DEFAULT, 5, a, b, c, budget)
    lt = 64 << 20
    # square tiles: the same plan as himuon_ns_gemm
    assert ws([1024], [1024], 512, 512) == hm.himuon_ns_gemm_workspace_size([1024], [1024], 512, hm.BF16, 0, 5, a, b, c)
    # a tall and a wide tile of the same size are one (m, n) problem shape: the same workspace
    assert ws([1024], [1024], 256, 128) == ws([1024], [1024], 128, 256) > lt
    # 32 tiles of 128 x 256: X, X' (128 x 256) and A, B (128 x 128) in fp16 per tile
    need = ws([1024], [1024], 128, 256)
    assert need >= lt + 32 * (2 * 128 * 256 + 2 * 128 * 128) * 2
    # one tile covering the matrix is the whole matrix: the T = 0 plan
    assert ws([300], [500], 512, 600) == ws([300], [500], 0, 0)
    # exactly one of Th, Tw zero, or negative, has no plan
    assert ws([64], [64], 0, 64) == 0 and ws([64], [64], 64, 0) == 0 and ws([64], [64], -1, 64) == 0
    args = dict(n_mats=1, in_ptrs=[FAKE], out_ptrs=[FAKE], rows=[64], cols=[64], ld_in=None, ld_out=None, Th=0, Tw=32,
                K=5, a=a, b=b, c=c, dtype=hm.BF16, compute=hm.COMPUTE_DEFAULT, workspace=FAKE, workspace_bytes=256,
                chunk_budget_bytes=0, stream=None)
    assert hm.himuon_ns_gemm_hw(**args) == hm.ERR_INVALID_ARG
    args.update(Th=32, Tw=64)
    assert hm.himuon_ns_gemm_hw(**args) == hm.ERR_WORKSPACE


@pytest.mark.parametrize("args", [
    (hm.COMPUTE_F16, 0, FAKE, 1, 1),        # no operands
    (hm.COMPUTE_F16, FAKE, 0, 1, 1),        # no output
    (hm.COMPUTE_F16, FAKE, FAKE, 0, 1),     # empty grid
    (hm.COMPUTE_F16, FAKE, FAKE, (1 << 20) + 1, 1),  # lane indices past int range
    (hm.COMPUTE_BF16, FAKE, FAKE, 1, 0),    # no products
    (hm.COMPUTE_F32, FAKE, FAKE, 1, 1),     # fp32 operands: no such calibration
    (hm.COMPUTE_DEFAULT, FAKE, FAKE, 1, 1),
])
def test_calib_mfma_rejects_bad_arguments_before_any_launch(args):
    assert hm.himuon_calib_mfma(*args) == hm.ERR_INVALID_ARG
