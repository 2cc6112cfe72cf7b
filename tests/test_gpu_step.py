"""The optimizer step (himuon_step, Alg. 1) against the fp64 oracle's step.

All three routes are covered: the library-GEMM path (T = 0, the
full-matrix branch, and T = 512) with the momentum fused into its gather and
the update into its scatter; the step inside the fused tile kernels (T = 128,
64, 32: bf16 with fp16 or bf16 operands, fp32); and the fused tile kernels
with element-wise prologue and epilogue (T = 256; c = 0). Bars:
  - momentum M: each element within one unit in the last place of the
    storage type of the oracle's value (the GPU rounds beta M + G once to
    storage; the oracle keeps fp64);
  - weights W: per tile, ||W_gpu - W_ref|| <= tol * ||lr tau U_ref|| +
    u * ||W_ref||, with tol the tiled map's bar (1e-5 fp32, 2e-2 bf16) on the
    direction and u the storage type's unit roundoff (2^-24, 2^-8) for the
    final rounding of W;
  - the direction itself, read back as (W_gpu - (1 - lr lambda) W) / (-lr tau)
    with W = 0, per tile within the tiled map's bar;
  - pure decay (G = M = 0): W_gpu is exactly W rounded after one multiply.
The step's parameters (W ~ 0.05 N(0,1), lr = 0.1, lambda = 0.5) make both the
decay term lr lambda ||W|| and the update lr tau ||U|| at least ten times the
final rounding slack u ||W|| (u = 2^-8 for bf16), so that a step that dropped
either term fails the bound.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_27216_amd as hm
from parity import BF16_OPERAND_BAR, COEF32, TOL, tile_errors, to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
UNIT = {torch.float32: 2.0 ** -24, torch.bfloat16: 2.0 ** -8}
LR, WD, BETA, SC = 0.1, 0.5, 0.95, 0.2
W_SCALE = 0.05  # weights' entry scale
ULP = {torch.float32: 2.0 ** -23, torch.bfloat16: 2.0 ** -7}


def announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def rand(shape, dtype, seed, scale=1.0):
    g = np.random.default_rng(seed)
    x = g.standard_normal(shape) * scale
    return torch.tensor(x, dtype=torch.float32).to(dtype).to(DEV)


def f32(v):
    return float(np.float32(v))


def tau_of(H, W, T, sc):
    full = T == 0 or T >= max(H, W)
    return f32(sc) * np.sqrt(max(H, W) if full else T)


def check_step(W0, G, M0, W1, M1, T, dtype, lr, beta, wd, nesterov, sc, K=5, tile=None, tol=None):
    """W0, G, M0: the inputs (device); W1, M1: the GPU's results; `tol` the
    bar on the direction (default: the tiled map's bar for `dtype`)."""
    tol = TOL[dtype] if tol is None else tol
    Wr, Mr, Ur = oracle.himuon_step(to_f64(W0), to_f64(M0), to_f64(G), T, K, *COEF32, f32(lr), f32(beta), f32(wd),
                                    nesterov, f32(sc))
    m = to_f64(M1)
    # one rounding to storage, after fp32 arithmetic on beta M and G
    slack = 2.0 ** -22 * (f32(beta) * np.abs(to_f64(M0)) + np.abs(to_f64(G)))
    assert np.all(np.abs(m - Mr) <= ULP[dtype] * np.abs(Mr) + slack), \
        f"momentum off by more than one ulp: {np.max(np.abs(m - Mr) / (np.abs(Mr) + 1e-30)):.3e}"
    H, Wd = Wr.shape
    t = tile or (max(H, Wd) if T == 0 or T >= max(H, Wd) else T)
    upd = f32(lr) * tau_of(H, Wd, T, sc) * Ur
    w = to_f64(W1)
    worst = 0.0
    for r0 in range(0, H, t):
        for c0 in range(0, Wd, t):
            sl = np.s_[r0:r0 + t, c0:c0 + t]
            bound = tol * np.linalg.norm(upd[sl]) + UNIT[dtype] * np.linalg.norm(Wr[sl])
            err = np.linalg.norm(w[sl] - Wr[sl])
            assert err <= bound, f"tile ({r0},{c0}): |dW| {err:.3e} > {bound:.3e}"
            worst = max(worst, err / max(bound, 1e-300))
    return worst


def run_step(Ws, Gs, Ms, T, dtype, lr=LR, beta=BETA, wd=WD, nesterov=True, sc=SC, budget=0,
             compute=hm.COMPUTE_DEFAULT):
    hm.step(Ws, Gs, Ms, T=T, K=5, coeffs=COEF32, lr=lr, momentum=beta, weight_decay=wd, nesterov=nesterov,
            scale_c=sc, chunk_budget_bytes=budget, compute=compute)
    torch.cuda.synchronize()


def test_step_terms_exceed_rounding_slack():
    """The margin the bounds rely on (host arithmetic only): on a T x T tile
    with ||W|| = W_SCALE T and ||U|| >= 0.5 sqrt(T) (a converged tile has
    singular values near 1), decay and update are ten times the slack."""
    slack = UNIT[torch.bfloat16]
    assert LR * WD >= 10 * slack
    for T in (32, 64, 128, 256, 512):
        upd = LR * SC * np.sqrt(T) * 0.5 * np.sqrt(T)
        assert upd >= 10 * slack * W_SCALE * T


@pytest.mark.parametrize("T", [512, 0])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_gemm_route(T, dtype):
    shapes = [(700, 900), (520, 384), (64, 96)] if T else [(300, 500), (500, 300), (1, 257)]
    announce(f"step gemm route T={T} dtype={dtype} shapes={shapes}")
    W0 = [rand(s, dtype, 10 + i, W_SCALE) for i, s in enumerate(shapes)]
    G = [rand(s, dtype, 20 + i, 1e-2) for i, s in enumerate(shapes)]
    M0 = [rand(s, dtype, 30 + i, 1e-2) for i, s in enumerate(shapes)]
    W1 = [w.clone() for w in W0]
    M1 = [m.clone() for m in M0]
    run_step(W1, G, M1, T, dtype)
    for i in range(len(shapes)):
        check_step(W0[i], G[i], M0[i], W1[i], M1[i], T, dtype, LR, BETA, WD, True, SC)


@pytest.mark.parametrize("T", [128, 64, 32, 256])
@pytest.mark.parametrize("nesterov", [True, False])
def test_fused_route_bf16(T, nesterov):
    shapes = [(384, 520), (100, 60), (257, 131)]
    announce(f"step fused route T={T} nesterov={nesterov} bf16 shapes={shapes}")
    W0 = [rand(s, torch.bfloat16, 40 + i, W_SCALE) for i, s in enumerate(shapes)]
    G = [rand(s, torch.bfloat16, 50 + i, 1e-2) for i, s in enumerate(shapes)]
    M0 = [rand(s, torch.bfloat16, 60 + i, 1e-2) for i, s in enumerate(shapes)]
    W1 = [w.clone() for w in W0]
    M1 = [m.clone() for m in M0]
    run_step(W1, G, M1, T, torch.bfloat16, nesterov=nesterov)
    for i in range(len(shapes)):
        check_step(W0[i], G[i], M0[i], W1[i], M1[i], T, torch.bfloat16, LR, BETA, WD, nesterov, SC)


@pytest.mark.parametrize("T", [32, 64, 128, 256, 512, 0])
@pytest.mark.parametrize("mode", ["bf16/f16", "bf16/bf16", "f32"])
def test_direction_per_tile(T, mode):
    """W = 0, lambda = 0: the step leaves -lr tau U; U per tile within the
    map's bar, on every route (in the tile kernel: T = 32, 64, 128; around it:
    T = 256 with fp16 operands; the GEMM path: T = 512, 0, and T = 256 for
    fp32 storage or bf16 operands) and operand mode."""
    dtype = torch.float32 if mode == "f32" else torch.bfloat16
    compute = hm.COMPUTE_BF16 if mode == "bf16/bf16" else hm.COMPUTE_DEFAULT
    bar = BF16_OPERAND_BAR if mode == "bf16/bf16" else TOL[dtype]
    announce(f"step direction readback, T={T}, {mode}")
    H, Wd = (700, 900) if T != 0 else (300, 500)
    x = rand((H, Wd), dtype, 70, 1e-2)
    W = torch.zeros_like(x)
    M = torch.zeros_like(x)
    run_step([W], [x], [M], T, dtype, lr=0.5, beta=0.9, wd=0.0, compute=compute)
    _, _, Ur = oracle.himuon_step(np.zeros((H, Wd)), np.zeros((H, Wd)), to_f64(x), T, 5, *COEF32,
                                  f32(0.5), f32(0.9), 0.0, True, f32(SC))
    U = to_f64(W) / (-f32(0.5) * tau_of(H, Wd, T, SC))
    e = tile_errors(U, Ur, T if T else max(H, Wd))
    print(f"[gpu-err] direction T={T} {mode}: max {e.max():.3e}", flush=True)
    assert e.max() <= bar, f"T={T}: max per-tile error {e.max():.3e}"


@pytest.mark.parametrize("T", [32, 64, 128, 256, 512, 0])
@pytest.mark.parametrize("mode", ["bf16/f16", "bf16/bf16", "f32"])
def test_pure_decay_exact(T, mode):
    """G = M = 0, lr lambda = 0.25: Phi_K(0) = 0, so every route must leave
    exactly W (1 - lr lambda), rounded once to storage (0.75 W is exact in
    fp32), and M = 0."""
    dtype = torch.float32 if mode == "f32" else torch.bfloat16
    compute = hm.COMPUTE_BF16 if mode == "bf16/bf16" else hm.COMPUTE_DEFAULT
    announce(f"step pure decay, T={T}, {mode}")
    W = rand((300, 400), dtype, 140)
    W0 = W.clone()
    G = torch.zeros_like(W)
    M = torch.zeros_like(W)
    run_step([W], [G], [M], T, dtype, lr=0.5, wd=0.5, compute=compute)
    assert not torch.any(M)
    assert torch.equal(W, (W0.float() * 0.75).to(dtype))


@pytest.mark.parametrize("T", [512, 128])
def test_three_steps_fp32_with_reconfigure_keeping_momentum(T):
    """Three steps of the HiMuon state object (fp32), the second after a
    reconfigure to T = 0 and back: momentum carries across tile sizes."""
    announce(f"step x3 fp32 with reconfigure, T={T}")
    shape = (520, 700)
    p = rand(shape, torch.float32, 80)
    opt = hm.HiMuon([p], T=T, K=5, coeffs=COEF32, lr=0.05, momentum=0.9, weight_decay=0.05, nesterov=True,
                    scale_c=0.2)
    Wr, Mr = to_f64(p), np.zeros(shape)
    for t, Tt in enumerate([T, 0, T]):
        opt.reconfigure(Tt)
        g = rand(shape, torch.float32, 90 + t, 1e-2)
        W_before, M_before = p.clone(), opt.moms[0].clone()
        opt.step([g])
        torch.cuda.synchronize()
        check_step(W_before, g, M_before, p, opt.moms[0], Tt, torch.float32, 0.05, 0.9, 0.05, True, 0.2)
        Wr, Mr, _ = oracle.himuon_step(Wr, Mr, to_f64(g), Tt, 5, *COEF32, f32(0.05), f32(0.9), f32(0.05), True,
                                       f32(0.2))
    # the trajectory as a whole: three updates of size lr tau ~ 0.05 * 0.2 * sqrt(T)
    assert np.linalg.norm(to_f64(p) - Wr) <= 1e-5 * np.linalg.norm(Wr)
    assert np.linalg.norm(to_f64(opt.moms[0]) - Mr) <= 1e-6 * np.linalg.norm(Mr)


@pytest.mark.parametrize("T", [512, 128])
def test_state_object_on_a_side_stream(T):
    """HiMuon stepping on a stream of its own, with a reconfigure between
    steps (which may replace the cached workspace) and new allocations
    right after each step: the same bits as the same steps on the current
    stream."""
    announce(f"HiMuon on a side stream, T={T}, bf16")
    shapes = [(384, 512), (512, 384), (96, 1000)]
    P0 = [rand(s, torch.bfloat16, 140 + i, W_SCALE) for i, s in enumerate(shapes)]
    Gs = [[rand(s, torch.bfloat16, 150 + 10 * t + i, 1e-2) for i, s in enumerate(shapes)] for t in range(3)]

    def trajectory(stream):
        ps = [p.clone() for p in P0]
        opt = hm.HiMuon(ps, T=T, K=5, coeffs=COEF32, lr=0.05, momentum=0.9, weight_decay=0.1, tune=False)
        for t, Tt in enumerate([T, 0, T]):
            opt.reconfigure(Tt)
            if stream is None:
                opt.step(Gs[t])
            else:
                stream.wait_stream(torch.cuda.current_stream())  # the inputs were made on the current stream
                opt.step(Gs[t], stream=stream)
                # allocations on the current stream meanwhile, which must not get the workspace's memory
                junk = [torch.full((1 << 20,), 7.0, device=DEV) for _ in range(4)]
                del junk
        torch.cuda.synchronize()
        return ps, opt.moms

    side = torch.cuda.Stream(device=DEV)
    ref_p, ref_m = trajectory(None)
    got_p, got_m = trajectory(side)
    for a, b in zip(got_p + got_m, ref_p + ref_m):
        assert torch.equal(a, b)


@pytest.mark.parametrize("T", [512, 128])
def test_chunked_equals_unchunked(T):
    announce(f"step chunked vs one chunk, T={T}, bf16")
    shapes = [(1024, 1024), (512, 768), (640, 512)]
    W0 = [rand(s, torch.bfloat16, 100 + i, W_SCALE) for i, s in enumerate(shapes)]
    G = [rand(s, torch.bfloat16, 110 + i, 1e-2) for i, s in enumerate(shapes)]
    M0 = [rand(s, torch.bfloat16, 120 + i, 1e-2) for i, s in enumerate(shapes)]
    outs = []
    budget = 1024 * 1024 * 2 if T == 128 else 2 * (2 * 512 * 512 + 2 * 512 * 512) * 3
    for bud in (0, budget):
        W1 = [w.clone() for w in W0]
        M1 = [m.clone() for m in M0]
        run_step(W1, G, M1, T, torch.bfloat16, budget=bud)
        outs.append((W1, M1))
    # the momentum is element-wise either way
    for a, b in zip(outs[0][1], outs[1][1]):
        assert torch.equal(a, b)
    if T == 128:
        # fused route: groups of whole matrices, each tile's result is independent of its launch
        for a, b in zip(outs[0][0], outs[1][0]):
            assert torch.equal(a, b)
    else:
        # GEMM route: the GEMM library may pick another kernel for another batch count
        for i in range(len(shapes)):
            for W1 in (outs[0][0][i], outs[1][0][i]):
                check_step(W0[i], G[i], M0[i], W1, outs[0][1][i], T, torch.bfloat16, LR, BETA, WD, True, SC)


def test_non_contiguous_rows_and_untouched_gradient():
    """A row stride above the width (a column slice of a wider buffer); the
    gradient is read only, and the columns outside the slice stay as they were."""
    announce("step strided rows, T=128 and T=512, bf16")
    for T in (128, 512):
        big_w = rand((300, 720), torch.bfloat16, 130, W_SCALE)
        big_g = rand((300, 720), torch.bfloat16, 131, 1e-2)
        big_m = rand((300, 720), torch.bfloat16, 132, 1e-2)
        W, G, M = big_w[:, :600], big_g[:, :600], big_m[:, :600]
        W0, G0, M0 = W.clone(), G.clone(), M.clone()
        w_rest, g_all, m_rest = big_w[:, 600:].clone(), big_g.clone(), big_m[:, 600:].clone()
        run_step([W], [G], [M], T, torch.bfloat16)
        check_step(W0, G0, M0, W, M, T, torch.bfloat16, LR, BETA, WD, True, SC)
        assert torch.equal(big_g, g_all)
        assert torch.equal(big_w[:, 600:], w_rest) and torch.equal(big_m[:, 600:], m_rest)


@pytest.mark.parametrize("T", [128, 64, 32])
@pytest.mark.parametrize("nesterov", [True, False])
def test_in_kernel_route_fp32(T, nesterov):
    """fp32 storage: the step inside the generic tile kernel (fp32 operands)."""
    shapes = [(384, 520), (100, 60)]
    announce(f"step fp32 T={T} nesterov={nesterov} shapes={shapes}")
    W0 = [rand(s, torch.float32, 150 + i, W_SCALE) for i, s in enumerate(shapes)]
    G = [rand(s, torch.float32, 160 + i, 1e-2) for i, s in enumerate(shapes)]
    M0 = [rand(s, torch.float32, 170 + i, 1e-2) for i, s in enumerate(shapes)]
    W1 = [w.clone() for w in W0]
    M1 = [m.clone() for m in M0]
    run_step(W1, G, M1, T, torch.float32, nesterov=nesterov)
    for i in range(len(shapes)):
        check_step(W0[i], G[i], M0[i], W1[i], M1[i], T, torch.float32, LR, BETA, WD, nesterov, SC)


def test_in_kernel_route_bf16_operands():
    """bf16 storage with bf16 MFMA operands: the step inside the generic kernel."""
    shapes = [(384, 520), (100, 60)]
    announce(f"step bf16 operands T=128 shapes={shapes}")
    W0 = [rand(s, torch.bfloat16, 190 + i, W_SCALE) for i, s in enumerate(shapes)]
    G = [rand(s, torch.bfloat16, 191 + i, 1e-2) for i, s in enumerate(shapes)]
    M0 = [rand(s, torch.bfloat16, 192 + i, 1e-2) for i, s in enumerate(shapes)]
    W1 = [w.clone() for w in W0]
    M1 = [m.clone() for m in M0]
    run_step(W1, G, M1, 128, torch.bfloat16, compute=hm.COMPUTE_BF16)
    for i in range(len(shapes)):
        check_step(W0[i], G[i], M0[i], W1[i], M1[i], 128, torch.bfloat16, LR, BETA, WD, True, SC,
                   tol=BF16_OPERAND_BAR)


def test_prologue_epilogue_route_c_zero():
    """c = 0 (the cubic (1.5, -0.5, 0)) at T = 128, bf16: the fp16 kernel has no
    step variant for it, so the element-wise prologue and epilogue run around it."""
    cubic = (1.5, -0.5, 0.0)
    shapes = [(300, 200)]
    announce("step c = 0 bf16 T=128 (prologue/epilogue)")
    W0 = [rand(s, torch.bfloat16, 195, W_SCALE) for s in shapes]
    G = [rand(s, torch.bfloat16, 196, 1e-2) for s in shapes]
    M0 = [rand(s, torch.bfloat16, 197, 1e-2) for s in shapes]
    W1 = [w.clone() for w in W0]
    M1 = [m.clone() for m in M0]
    hm.step(W1, G, M1, T=128, K=5, coeffs=cubic, lr=LR, momentum=BETA, weight_decay=WD, nesterov=True,
            scale_c=SC)
    torch.cuda.synchronize()
    Wr, Mr, Ur = oracle.himuon_step(to_f64(W0[0]), to_f64(M0[0]), to_f64(G[0]), 128, 5, *cubic, f32(LR),
                                    f32(BETA), f32(WD), True, f32(SC))
    upd = f32(LR) * tau_of(300, 200, 128, SC) * Ur
    for r0 in range(0, 300, 128):
        for c0 in range(0, 200, 128):
            sl = np.s_[r0:r0 + 128, c0:c0 + 128]
            err = np.linalg.norm(to_f64(W1[0])[sl] - Wr[sl])
            assert err <= 2e-2 * np.linalg.norm(upd[sl]) + 2.0 ** -8 * np.linalg.norm(Wr[sl])


def _p_iter(K, s=1.0):
    a, b, c = COEF32
    for _ in range(K):
        s = a * s + b * s ** 3 + c * s ** 5
    return s


@pytest.mark.parametrize("T,dtype", [(128, torch.float32), (0, torch.float32), (128, torch.bfloat16)])
def test_more_matrices_than_one_grid_row(T, dtype):
    """70,000 matrices of 1 x 8 in one call: more than the 65,535 a launch
    covers per grid row (the element-wise kernels and the GEMM path split
    them). Each is rank one, so Phi_K(G) = p^K(1) G / ||G|| with one tau =
    c sqrt(8) (T >= max(H, W): the full branch); the oracle checks a sample."""
    n = 70000
    announce(f"step with {n} matrices of 1x8, T={T}, {dtype}")
    W = rand((n, 8), dtype, 180)
    G = rand((n, 8), dtype, 181, 1e-2)
    M = torch.zeros_like(W)
    W0 = W.clone()
    Ws, Gs, Ms = [W[i:i + 1] for i in range(n)], [G[i:i + 1] for i in range(n)], [M[i:i + 1] for i in range(n)]
    run_step(Ws, Gs, Ms, T, dtype, lr=0.05, beta=0.9, wd=0.0)
    g = to_f64(G)
    mm = f32(0.9) * 0 + g                       # M = 0 + G
    gh = g + f32(0.9) * to_f64(M)               # Nesterov lookahead from the stored M
    assert np.allclose(to_f64(M), mm, rtol=ULP[dtype], atol=0)
    U = _p_iter(5) * gh / np.linalg.norm(gh, axis=1, keepdims=True)
    ref = to_f64(W0) - f32(0.05) * f32(0.2) * np.sqrt(8.0) * U
    err = np.abs(to_f64(W) - ref).max(axis=1)
    bound = TOL[dtype] * f32(0.05) * f32(0.2) * np.sqrt(8.0) * np.abs(U).max(axis=1) + 2 * UNIT[dtype] * np.abs(ref).max(axis=1)
    assert np.all(err <= bound), f"worst row {int(np.argmax(err / bound))}: {np.max(err / bound):.3f} of the bar"
    for i in (0, 1, 65534, 65535, 65536, n - 1):
        check_step(W0[i:i + 1], G[i:i + 1], torch.zeros_like(W0[i:i + 1]), W[i:i + 1], M[i:i + 1], T, dtype, 0.05, 0.9,
                   0.0, True, 0.2)
