"""The fused rectangular-tile kernels (himuon_ns_tiled_hw) against the fp64
oracle's rectangular tiling (oracle.ns_tiled_hw), tile by tile.

Tiles are Th x Tw (the tile-shape study's fused region, Th Tw <= 16384); a
tall tile is iterated as its transpose, which the oracle does too. Bars as
for square tiles: 1e-5 (fp32 storage), 2e-2 (bf16 storage, fp16 operands),
the bf16-operand bar for bf16 operands; exact equality where the arithmetic
is the same (batching, chunking, in place).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_27216_amd as hm
import workloads
from parity import BF16_OPERAND_BAR, COEF32, TOL, to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
SHAPES_BF16 = [(32, 64), (32, 128), (32, 256), (32, 512), (64, 128), (64, 256)]
SHAPES_F32 = [(32, 64), (32, 128), (32, 256)]


def announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def rect_errors(Y, R, Th, Tw):
    H, W = R.shape
    errs = []
    for r0 in range(0, H, Th):
        for c0 in range(0, W, Tw):
            y, r = Y[r0:r0 + Th, c0:c0 + Tw], R[r0:r0 + Th, c0:c0 + Tw]
            n = np.linalg.norm(r)
            errs.append((0.0 if not np.any(y) else np.inf) if n == 0 else np.linalg.norm(y - r) / n)
    return np.array(errs)


def run(mats, Th, Tw, K=5, compute=hm.COMPUTE_DEFAULT, budget=0, outputs=None):
    out = hm.ns_tiled(mats, outputs=outputs, T=Th, Tw=Tw, K=K, coeffs=COEF32, compute=compute,
                      chunk_budget_bytes=budget)
    torch.cuda.synchronize()
    return out


def check(x, y, Th, Tw, K=5, bar=None):
    R = oracle.ns_tiled_hw(to_f64(x), Th, Tw, K, *COEF32)
    e = rect_errors(to_f64(y), R, Th, Tw)
    bar = TOL[x.dtype] if bar is None else bar
    assert np.all(np.isfinite(e)), "non-finite tile"
    print(f"[gpu-err] {tuple(x.shape)} {Th}x{Tw} K={K}: {len(e)} tiles, max {e.max():.3e} p50 {np.median(e):.3e}",
          flush=True)
    assert e.max() <= bar, f"{Th}x{Tw}: max per-tile error {e.max():.3e} > {bar:.1e}"
    return e


@pytest.mark.parametrize("dtype,shape", [("bf16", s) for s in SHAPES_BF16] + [("f32", s) for s in SHAPES_F32])
@pytest.mark.parametrize("tall", [False, True])
def test_rect_tiles_against_oracle(dtype, shape, tall):
    """A ragged batch (partial tiles on both edges, a matrix smaller than one
    tile) of heavy-tailed matrices, every tile against the oracle."""
    Th, Tw = (shape[1], shape[0]) if tall else shape
    mats = [workloads.student_t(3 * Th + 7, 2 * Tw + 19, 400 + Th + Tw, dtype, DEV),
            workloads.lowrank_plus_noise(5 * Th, 4 * Tw, 401, dtype, DEV),
            workloads.gaussian(Th // 2 + 1, Tw - 3, 402, dtype, DEV)]
    announce(f"rect {Th}x{Tw} {dtype} on {[tuple(m.shape) for m in mats]}")
    outs = run(mats, Th, Tw)
    for x, y in zip(mats, outs):
        check(x, y, Th, Tw)


@pytest.mark.parametrize("shape", [(32, 512), (64, 256), (256, 64)])
@pytest.mark.parametrize("K", [0, 1, 8])
def test_rect_step_counts(shape, K):
    Th, Tw = shape
    announce(f"rect {Th}x{Tw} bf16 K={K}")
    x = workloads.student_t(2 * Th + 5, 2 * Tw + 9, 410, "bf16", DEV)
    (y,) = run([x], Th, Tw, K=K)
    check(x, y, Th, Tw, K=K)


@pytest.mark.parametrize("shape", [(32, 256), (512, 32), (64, 128)])
def test_rect_bf16_operands(shape):
    Th, Tw = shape
    announce(f"rect {Th}x{Tw} bf16 operands")
    x = workloads.lowrank_plus_noise(4 * Th, 3 * Tw, 420, "bf16", DEV)
    (y,) = run([x], Th, Tw, compute=hm.COMPUTE_BF16)
    check(x, y, Th, Tw, bar=BF16_OPERAND_BAR)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_rect_batching_chunking_in_place_bitwise(dtype):
    Th, Tw = 32, 256
    announce(f"rect {Th}x{Tw} {dtype}: batched = alone = chunked = in place")
    mats = [workloads.student_t(h, w, 430 + i, dtype, DEV) for i, (h, w) in enumerate([(100, 700), (64, 256), (5, 3)])]
    base = run(mats, Th, Tw)
    for x, b in zip(mats, base):
        (alone,) = run([x], Th, Tw)
        assert torch.equal(alone, b)
    elem = 4 if dtype == "f32" else 2
    for tiles in (1, 3):
        for a, b in zip(run(mats, Th, Tw, budget=tiles * 2 * Th * Tw * elem), base):
            assert torch.equal(a, b)
    inplace = [m.clone() for m in mats]
    run(inplace, Th, Tw, outputs=inplace)
    for a, b in zip(inplace, base):
        assert torch.equal(a, b)


def test_rect_zero_tile_and_scale():
    Th, Tw = 64, 128
    announce(f"rect {Th}x{Tw} bf16: zero tile, 2^e scale")
    x = workloads.gaussian(2 * Th, 2 * Tw, 440, "bf16", DEV)
    x[:Th, Tw:] = 0
    (y,) = run([x], Th, Tw)
    assert not torch.any(y[:Th, Tw:])
    for e in (-30, 7):
        (z,) = run([x * (2.0 ** e)], Th, Tw)
        assert torch.equal(z, y), e


def test_rect_square_is_the_square_call_and_unsupported_shapes():
    x = workloads.gaussian(300, 200, 450, "bf16", DEV)
    a = run([x], 64, 64)
    b = hm.ns_tiled([x], T=64, K=5, coeffs=COEF32)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0])
    for Th, Tw in ((16, 1024), (128, 256), (64, 512)):
        with pytest.raises(hm.HimuonError) as err:
            run([x], Th, Tw)
        assert err.value.status == hm.ERR_UNSUPPORTED
    xf = workloads.gaussian(300, 200, 451, "f32", DEV)
    with pytest.raises(hm.HimuonError) as err:
        run([xf], 64, 128)
    assert err.value.status == hm.ERR_UNSUPPORTED


def test_rect_agrees_with_library_gemm_path():
    Th, Tw = 256, 64
    announce("rect 256x64 fused vs library GEMMs, bf16")
    x = workloads.lowrank_plus_noise(700, 900, 460, "bf16", DEV)
    (y,) = run([x], Th, Tw)
    (z,) = hm.ns_gemm([x], T=Th, Tw=Tw, K=5, coeffs=COEF32)
    torch.cuda.synchronize()
    e = rect_errors(to_f64(y), to_f64(z), Th, Tw)
    assert e.max() <= 2e-2, e.max()
