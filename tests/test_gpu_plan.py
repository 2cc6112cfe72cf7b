"""Plans (himuon_plan_*): a call recorded into a HIP graph and replayed.

Each replay must equal the recorded call run eagerly on the same buffer
contents, bit for bit. Between replays the program does its own eager work
on the same stream (new gradients or inputs are written into the recorded
buffers) and synchronises, and every replay is checked, so a graph node that
misbehaves on replays after the first cannot hide.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_27216_amd as hm
import workloads
from parity import COEF32, TOL, tile_errors, to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
SHAPES = [(384, 520), (1024, 1024), (100, 60)]


def announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def fill(ts, gen, scale):
    for t in ts:
        t.copy_((torch.randn(t.shape, device=DEV, generator=gen) * scale).to(t.dtype))


@pytest.mark.parametrize("T,dtype", [(128, "bf16"), (64, "f32"), (256, "bf16"), (512, "bf16"), (0, "f32")])
def test_step_plan_replays_equal_eager_steps(T, dtype):
    """The recorded optimizer step, on each route (inside the tile kernel,
    prologue/epilogue around it, library GEMMs), against eager himuon_step."""
    announce(f"step plan T={T} {dtype}, 4 replays")
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    gen = torch.Generator(device=DEV)
    gen.manual_seed(T + 7)
    W = [(torch.randn(s, device=DEV, generator=gen) * 0.05).to(tdt) for s in SHAPES]
    G = [torch.zeros(s, dtype=tdt, device=DEV) for s in SHAPES]
    W_ref = [w.clone() for w in W]
    M_ref = [torch.zeros_like(w) for w in W]
    opt = hm.HiMuon(W, T=T, K=5, coeffs=COEF32, lr=0.1, momentum=0.95, weight_decay=0.5, nesterov=True,
                    scale_c=0.2, capture=True, tune=False)
    for it in range(4):
        fill(G, gen, 1e-2)
        opt.step(G)
        hm.step(W_ref, G, M_ref, T=T, K=5, coeffs=COEF32, lr=0.1, momentum=0.95, weight_decay=0.5, nesterov=True,
                scale_c=0.2)
        torch.cuda.synchronize()
        for a, b in zip(W, W_ref):
            assert torch.equal(a, b), f"replay {it}: weights differ"
        for a, b in zip(opt.moms, M_ref):
            assert torch.equal(a, b), f"replay {it}: momenta differ"


def test_step_plan_follows_reconfigure():
    """reconfigure(T) drops the recorded step; the next step records the new
    tile size, and the momentum carries over."""
    announce("step plan with reconfigure 128 -> 512 -> 128, bf16")
    gen = torch.Generator(device=DEV)
    gen.manual_seed(11)
    W = [(torch.randn(s, device=DEV, generator=gen) * 0.05).to(torch.bfloat16) for s in SHAPES]
    G = [torch.zeros(s, dtype=torch.bfloat16, device=DEV) for s in SHAPES]
    W_ref = [w.clone() for w in W]
    M_ref = [torch.zeros_like(w) for w in W]
    opt = hm.HiMuon(W, T=128, K=5, coeffs=COEF32, lr=0.1, momentum=0.9, weight_decay=0.5, capture=True, tune=False)
    for it, T in enumerate((128, 512, 128)):
        opt.reconfigure(T)
        fill(G, gen, 1e-2)
        opt.step(G)
        hm.step(W_ref, G, M_ref, T=T, K=5, coeffs=COEF32, lr=0.1, momentum=0.9, weight_decay=0.5)
        torch.cuda.synchronize()
        for a, b in zip(W, W_ref):
            assert torch.equal(a, b), f"step {it} (T={T}): weights differ"


@pytest.mark.parametrize("T,dtype", [(128, "bf16"), (32, "bf16"), (256, "f32")])
def test_ns_tiled_plan_replays(T, dtype):
    """The recorded map on new input contents at every replay: equal to the
    eager call, and within the oracle's bar."""
    announce(f"ns_tiled plan T={T} {dtype}, 3 replays")
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    gen = torch.Generator(device=DEV)
    gen.manual_seed(T)
    X = [torch.zeros(s, dtype=tdt, device=DEV) for s in SHAPES]
    Y = [torch.empty_like(x) for x in X]
    plan = hm.plan_ns_tiled(X, Y, T=T, K=5, coeffs=COEF32)
    for it in range(3):
        fill(X, gen, 1.0)
        plan.launch()
        ref = hm.ns_tiled(X, T=T, K=5, coeffs=COEF32)
        torch.cuda.synchronize()
        for x, y, r in zip(X, Y, ref):
            assert torch.equal(y, r), f"replay {it}: output differs from the eager call"
        e = tile_errors(to_f64(Y[0]), oracle.ns_tiled(to_f64(X[0]), T, 5, *COEF32), T)
        assert e.max() <= TOL[tdt], e.max()
    plan.close()


@pytest.mark.parametrize("T,dtype", [(512, "bf16"), (0, "f32"), (0, "bf16")])
def test_ns_gemm_plan_replays(T, dtype):
    """The recorded library-GEMM call (large tiles, or whole matrices for
    T = 0): every replay on new input contents equals the eager call, and
    stays within the oracle's bar."""
    announce(f"ns_gemm plan T={T} {dtype}, 3 replays")
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    gen = torch.Generator(device=DEV)
    gen.manual_seed(T + 3)
    shapes = [(600, 1100), (1024, 512), (100, 60)]
    X = [torch.zeros(s, dtype=tdt, device=DEV) for s in shapes]
    Y = [torch.empty_like(x) for x in X]
    plan = hm.plan_ns_gemm(X, Y, T=T, K=5, coeffs=COEF32)
    for it in range(3):
        fill(X, gen, 1.0)
        plan.launch()
        ref = hm.ns_gemm(X, T=T, K=5, coeffs=COEF32)
        torch.cuda.synchronize()
        for y, r in zip(Y, ref):
            assert torch.equal(y, r), f"replay {it}: output differs from the eager call"
        x0, y0 = to_f64(X[0]), to_f64(Y[0])
        if T == 0:
            R = oracle.phi_k(x0, 5, *COEF32)
            e = np.array([np.linalg.norm(y0 - R) / np.linalg.norm(R)])
        else:
            e = tile_errors(y0, oracle.ns_tiled(x0, T, 5, *COEF32), T)
        assert e.max() <= TOL[tdt], e.max()
    plan.close()


def test_plan_rejects_bad_arguments_and_foreign_streams():
    x = workloads.gaussian(64, 64, 1, "bf16", DEV)
    ws = torch.empty(256, dtype=torch.uint8, device=DEV)
    st, h = hm.himuon_plan_ns_tiled(1, [x.data_ptr()], [x.data_ptr()], [64], [64], None, None, 48, 5, *COEF32,
                                    hm.BF16, hm.COMPUTE_DEFAULT, ws.data_ptr(), 256, 0)
    assert st == hm.ERR_UNSUPPORTED and h is None
    st, h = hm.himuon_plan_ns_tiled(1, [x.data_ptr()], [x.data_ptr()], [64], [64], None, None, 32, 5, *COEF32,
                                    hm.BF16, hm.COMPUTE_DEFAULT, ws.data_ptr(), 16, 0)
    assert st == hm.ERR_WORKSPACE and h is None
    assert hm.himuon_plan_launch(None, None) == hm.ERR_INVALID_ARG
