"""Pins that tie the fp64 oracle to the mathematics, not to itself.

Each ``pin_*`` function runs the oracle (optionally a library built from a
mutated copy of its source) on inputs whose exact answer follows from the
paper's definitions by an independent route, and returns the largest
relative error it saw. The routes:

* the SVD closed form: X X^T = U Σ² U^T, so every step of eq. (ns_iteration)
  maps each singular value s to p(s) = a s + b s³ + c s⁵ and keeps U, V;
  Φ_K(S) = U · diag(p^∘K(σ_i/‖S‖_F)) · V^T  (LAPACK ``dgesdd`` via numpy);
* exact rational arithmetic (``fractions``) for p^∘K at rank-1, diagonal,
  1×1 and scaled-orthogonal inputs;
* the tiling operator of Sec. 2.1 applied with numpy slicing, each block then
  checked against the SVD closed form (zero padding leaves Φ_K unchanged,
  Sec. 4.4.3: padded rows and columns stay zero and do not change the norm);
* invariances that any correct implementation obeys: transposition,
  orthogonal equivariance, odd homogeneity of degree 0, tile permutation;
* the textbook special case: cubic Newton–Schulz (1.5, −0.5, 0) converges to
  the polar factor (``scipy.linalg.polar``) for well-conditioned input;
* rectangular tiles: the same slicing with T_h x T_w blocks;
* for the optimizer step of Alg. 1: geometric sums over repeated steps with a
  constant gradient (the momentum buffer and the decayed weights have closed
  forms, and Φ_K is blind to positive scaling), the sign of the second
  update under a gradient that reverses, and the branch rule of eq.
  (scaled_update) on shapes where tiling and the full map give different τ.

``run_all`` is used by the mutation test in a subprocess, so a mutant that
crashes or misbehaves anywhere is reported as caught.
"""
from __future__ import annotations

import sys
from fractions import Fraction

import numpy as np
import scipy.linalg

import oracle

QUINTIC = (3.4445, -4.7750, 2.0315)  # eq. (ns_quintic)
TOL = 1e-10


def p_exact(s: Fraction, K: int, a=QUINTIC[0], b=QUINTIC[1], c=QUINTIC[2]) -> Fraction:
    """p^∘K(s) in exact rational arithmetic with the decimal coefficients."""
    a, b, c = Fraction(str(a)), Fraction(str(b)), Fraction(str(c))
    for _ in range(K):
        s = a * s + b * s ** 3 + c * s ** 5
    return s


def p_float(s, K, a=QUINTIC[0], b=QUINTIC[1], c=QUINTIC[2]):
    s = np.asarray(s, dtype=np.float64).copy()
    for _ in range(K):
        s = a * s + b * s ** 3 + c * s ** 5
    return s


def svd_closed_form(S, K, a=QUINTIC[0], b=QUINTIC[1], c=QUINTIC[2]):
    S = np.asarray(S, dtype=np.float64)
    n = np.linalg.norm(S)
    if n == 0.0:
        return np.zeros_like(S)
    U, s, Vt = np.linalg.svd(S, full_matrices=False)
    return (U * p_float(s / n, K, a, b, c)) @ Vt


def rel(X, Y):
    d = np.linalg.norm(np.asarray(X) - np.asarray(Y))
    n = np.linalg.norm(np.asarray(Y))
    return d / n if n > 0 else d


def pin_svd_closed_form(lib=None):
    """Φ_K on square, wide and tall matrices equals the SVD closed form."""
    rng = np.random.default_rng(11)
    err = 0.0
    for (H, W, K) in [(5, 5, 5), (7, 3, 5), (3, 8, 5), (32, 32, 5), (17, 40, 8), (40, 17, 3), (16, 16, 0)]:
        S = rng.standard_normal((H, W))
        err = max(err, rel(oracle.phi_k(S, K, *QUINTIC, lib=lib), svd_closed_form(S, K)))
    # arbitrary coefficients too (the library takes a, b, c as arguments)
    S = rng.standard_normal((9, 12))
    coef = (2.0, -1.5, 0.5)
    err = max(err, rel(oracle.phi_k(S, 4, *coef, lib=lib), svd_closed_form(S, 4, *coef)))
    return err


def pin_tiled_blocks(lib=None):
    """Φ_{K,T} on ragged matrices equals the closed form of every h×w block
    cut by numpy slicing (grid anchored at (0,0), padding at bottom/right)."""
    rng = np.random.default_rng(12)
    err = 0.0
    for (H, W, T, K) in [(70, 100, 32, 5), (33, 9, 8, 5), (64, 64, 16, 3), (5, 50, 16, 8)]:
        S = rng.standard_normal((H, W))
        Y = oracle.ns_tiled(S, T, K, *QUINTIC, lib=lib)
        for r0 in range(0, H, T):
            for c0 in range(0, W, T):
                blk = S[r0:r0 + T, c0:c0 + T]
                err = max(err, rel(Y[r0:r0 + T, c0:c0 + T], svd_closed_form(blk, K)))
    return err


def pin_sampled_tiles(lib=None):
    """The per-tile entry point returns the padded T×T tile: block in the
    top-left corner equal to the closed form, zeros elsewhere."""
    rng = np.random.default_rng(13)
    H, W, T, K = 45, 70, 32, 5
    S = rng.standard_normal((H, W))
    ids = [0, 1, 2, 3]
    Y = oracle.ns_tiles(S, T, K, *QUINTIC, ids, lib=lib)
    err = 0.0
    C = -(-W // T)
    for s, t in enumerate(ids):
        r, c = divmod(t, C)
        blk = S[r * T:(r + 1) * T, c * T:(c + 1) * T]
        h, w = blk.shape
        exp = np.zeros((T, T))
        exp[:h, :w] = svd_closed_form(blk, K)
        err = max(err, rel(Y[s], exp))
        if h < T or w < T:  # padding must come back exactly zero
            pad = Y[s].copy()
            pad[:h, :w] = 0.0
            err = max(err, float(np.abs(pad).max()))
    return err


def pin_rank_one(lib=None):
    """S = σ u v^T ⇒ Φ_K(S) = p^∘K(1) · S/‖S‖_F, p^∘K(1) exact rational."""
    rng = np.random.default_rng(14)
    err = 0.0
    for (n, m, K) in [(32, 32, 5), (8, 20, 8), (20, 8, 5)]:
        u = rng.standard_normal(n)
        v = rng.standard_normal(m)
        S = 3.7 * np.outer(u, v)
        exp = float(p_exact(Fraction(1), K)) * S / np.linalg.norm(S)
        err = max(err, rel(oracle.phi_k(S, K, *QUINTIC, lib=lib), exp))
    return err


def pin_scaled_orthogonal(lib=None):
    """S = αQ (T×T orthogonal) ⇒ Φ_K(S) = p^∘K(1/√T)·Q, since every singular
    value of S/‖S‖_F is 1/√T. Exercised through the tiled entry point with
    one full tile."""
    rng = np.random.default_rng(15)
    err = 0.0
    for T in (4, 16, 32):
        Q, _ = np.linalg.qr(rng.standard_normal((T, T)))
        S = 0.125 * Q
        for K in (5, 8):
            # p^∘K(1/√T) with 1/√T irrational: use the float closed form
            exp = p_float(1.0 / np.sqrt(T), K) * Q
            err = max(err, rel(oracle.ns_tiled(S, T, K, *QUINTIC, lib=lib), exp))
    return err


def pin_diagonal(lib=None):
    """diag(3, 4) has ‖·‖_F = 5, so Φ_K = diag(p^∘K(3/5), p^∘K(4/5)) exactly;
    a 1×1 tile [s] gives sign(s)·p^∘K(1)."""
    err = 0.0
    for K in (1, 2, 5):
        Y = oracle.phi_k(np.array([[3.0, 0.0], [0.0, 4.0]]), K, *QUINTIC, lib=lib)
        exp = np.array([[float(p_exact(Fraction(3, 5), K)), 0.0], [0.0, float(p_exact(Fraction(4, 5), K))]])
        err = max(err, rel(Y, exp))
        # an anti-diagonal arrangement (a permutation of the same singular values)
        Y = oracle.phi_k(np.array([[0.0, -3.0], [4.0, 0.0]]), K, *QUINTIC, lib=lib)
        exp = np.array([[0.0, -float(p_exact(Fraction(3, 5), K))], [float(p_exact(Fraction(4, 5), K)), 0.0]])
        err = max(err, rel(Y, exp))
    for s in (-2.5, 0.75):
        Y = oracle.ns_tiled(np.array([[s]]), 1, 5, *QUINTIC, lib=lib)
        err = max(err, rel(Y, np.array([[np.sign(s) * float(p_exact(Fraction(1), 5))]])))
    return err


def pin_zero(lib=None):
    """Φ_K(0) = 0 (Sec. 2.2); a zero tile inside a nonzero matrix stays zero
    and its neighbours are unaffected."""
    S = np.zeros((40, 40))
    Y = oracle.ns_tiled(S, 16, 5, *QUINTIC, lib=lib)
    err = float(np.abs(Y).max())
    rng = np.random.default_rng(16)
    S = rng.standard_normal((32, 48))
    S[0:16, 16:32] = 0.0
    Y = oracle.ns_tiled(S, 16, 5, *QUINTIC, lib=lib)
    err = max(err, float(np.abs(Y[0:16, 16:32]).max()))
    err = max(err, rel(Y[16:32, 32:48], svd_closed_form(S[16:32, 32:48], 5)))
    return err


def pin_special_coefficients(lib=None):
    """K = 0 or (a,b,c) = (1,0,0) give S/‖S‖_F; (0,1,0) cubes the singular
    values K times (s ↦ s^(3^K))."""
    rng = np.random.default_rng(17)
    S = rng.standard_normal((12, 20))
    N = S / np.linalg.norm(S)
    err = rel(oracle.phi_k(S, 0, *QUINTIC, lib=lib), N)
    err = max(err, rel(oracle.phi_k(S, 6, 1.0, 0.0, 0.0, lib=lib), N))
    U, s, Vt = np.linalg.svd(N, full_matrices=False)
    err = max(err, rel(oracle.phi_k(S, 2, 0.0, 1.0, 0.0, lib=lib), (U * s ** 9) @ Vt))
    return err


def pin_cubic_polar(lib=None):
    """Textbook cubic Newton–Schulz X ← 1.5X − 0.5XX^TX converges to the polar
    factor polar(S) = UV^T for full-rank input (Sec. 2.2)."""
    rng = np.random.default_rng(18)
    err = 0.0
    for (n, m) in [(8, 8), (6, 10)]:
        U, _ = np.linalg.qr(rng.standard_normal((n, n)))
        V, _ = np.linalg.qr(rng.standard_normal((m, n)))
        S = (U * np.linspace(1.0, 4.0, n)) @ V.T  # condition number 4
        if n == m:
            P, _ = scipy.linalg.polar(S)
        else:
            P = U @ V.T
        err = max(err, rel(oracle.phi_k(S, 60, 1.5, -0.5, 0.0, lib=lib), P))
    return err


def pin_invariances(lib=None):
    """Transposition Φ(S^T) = Φ(S)^T, equivariance Φ(PSQ) = PΦ(S)Q, and
    Φ(αS) = sign(α)Φ(S)."""
    rng = np.random.default_rng(19)
    S = rng.standard_normal((16, 16))
    Y = oracle.phi_k(S, 5, *QUINTIC, lib=lib)
    err = rel(oracle.phi_k(S.T, 5, *QUINTIC, lib=lib), Y.T)
    R = rng.standard_normal((10, 24))
    err = max(err, rel(oracle.phi_k(R.T, 5, *QUINTIC, lib=lib), oracle.phi_k(R, 5, *QUINTIC, lib=lib).T))
    P, _ = np.linalg.qr(rng.standard_normal((16, 16)))
    Q, _ = np.linalg.qr(rng.standard_normal((16, 16)))
    err = max(err, rel(oracle.phi_k(P @ S @ Q, 5, *QUINTIC, lib=lib), P @ Y @ Q))
    err = max(err, rel(oracle.phi_k(-1e-3 * S, 5, *QUINTIC, lib=lib), -Y))
    err = max(err, rel(oracle.phi_k(2.0 ** 40 * S, 5, *QUINTIC, lib=lib), Y))
    return err


def pin_tile_permutation(lib=None):
    """Tiles are independent: permuting the tiles of the input permutes the
    tiles of Φ_{K,T} the same way (Sec. 4.4.2, cross-layer batching)."""
    rng = np.random.default_rng(20)
    T, R, C = 8, 3, 4
    S = rng.standard_normal((R * T, C * T))
    Y = oracle.ns_tiled(S, T, 5, *QUINTIC, lib=lib)
    perm = rng.permutation(R * C)
    Sp = np.empty_like(S)
    Yp = np.empty_like(S)
    for dst, src in enumerate(perm):
        (dr, dc), (sr, sc) = divmod(dst, C), divmod(src, C)
        Sp[dr * T:(dr + 1) * T, dc * T:(dc + 1) * T] = S[sr * T:(sr + 1) * T, sc * T:(sc + 1) * T]
        Yp[dr * T:(dr + 1) * T, dc * T:(dc + 1) * T] = Y[sr * T:(sr + 1) * T, sc * T:(sc + 1) * T]
    return rel(oracle.ns_tiled(Sp, T, 5, *QUINTIC, lib=lib), Yp)


def pin_single_tile_is_full_map(lib=None):
    """T ≥ max(H, W) gives one padded tile and Φ_{K,T} = Φ_K (Sec. 4.4.3);
    T = H = W is full-matrix Muon Newton–Schulz."""
    rng = np.random.default_rng(21)
    S = rng.standard_normal((24, 24))
    err = rel(oracle.ns_tiled(S, 24, 5, *QUINTIC, lib=lib), svd_closed_form(S, 5))
    R = rng.standard_normal((13, 29))
    err = max(err, rel(oracle.ns_tiled(R, 32, 5, *QUINTIC, lib=lib), svd_closed_form(R, 5)))
    err = max(err, rel(oracle.ns_tiled(R.T, 32, 5, *QUINTIC, lib=lib), svd_closed_form(R.T, 5)))
    return err


def pin_tile_count(lib=None):
    """R·C with ceilings (eq. tiling_operator); returns 0 when all agree."""
    bad = 0
    for (H, W, T) in [(256, 256, 32), (70, 100, 32), (1, 1, 128), (11008, 4096, 128), (129, 4096, 128)]:
        bad += oracle.tile_count(H, W, T, lib=lib) != (-(-H // T)) * (-(-W // T))
    return float(bad)


def pin_rect_tiled_blocks(lib=None):
    """Rectangular tiles (the tile-shape study): pad to (R T_h) x (C T_w) by
    numpy, cut T_h x T_w blocks, each by the SVD closed form (which needs no
    orientation choice); tall and wide tiles, ragged edges, and one tile
    covering the matrix (the full map)."""
    g = np.random.default_rng(31)
    worst = 0.0
    for (H, W, Th, Tw) in [(100, 150, 32, 64), (100, 150, 64, 16), (70, 45, 48, 48), (37, 90, 40, 100),
                           (90, 37, 16, 8)]:
        S = g.standard_normal((H, W))
        Y = oracle.ns_tiled_hw(S, Th, Tw, 5, *QUINTIC, lib=lib)
        R, C = -(-H // Th), -(-W // Tw)
        P = np.zeros((R * Th, C * Tw))
        P[:H, :W] = S
        Ref = np.zeros_like(P)
        for r in range(R):
            for q in range(C):
                blk = np.s_[r * Th:(r + 1) * Th, q * Tw:(q + 1) * Tw]
                Ref[blk] = svd_closed_form(P[blk], 5)
        worst = max(worst, rel(Y, Ref[:H, :W]))
    return worst


STEP = dict(a=QUINTIC[0], b=QUINTIC[1], c=QUINTIC[2], K=5)


def _tilewise_closed_form(S, T, K):
    """Φ_{K,T} by numpy slicing of the zero-padded matrix, each tile by SVD."""
    H, W = S.shape
    R, C = -(-H // T), -(-W // T)
    P = np.zeros((R * T, C * T))
    P[:H, :W] = S
    Y = np.zeros_like(P)
    for r in range(R):
        for q in range(C):
            Y[r * T:(r + 1) * T, q * T:(q + 1) * T] = svd_closed_form(P[r * T:(r + 1) * T, q * T:(q + 1) * T], K)
    return Y[:H, :W]


def pin_step_constant_gradient(lib=None):
    """t steps from M = 0 with one gradient G: M_t = G (1 - β^t)/(1 - β); the
    direction Ĝ is a positive multiple of G (either flag), so U = Φ_{K,T}(G)
    every step and W_t = d^t W_0 - lr τ U (1 - d^t)/(1 - d), d = 1 - lr λ."""
    g = np.random.default_rng(21)
    worst = 0.0
    lr, beta, lam, sc, steps = 0.05, 0.9, 0.3, 0.2, 4
    for (H, W, T, nesterov) in [(48, 100, 32, True), (48, 100, 64, False), (90, 60, 0, True), (33, 33, 128, False)]:
        G = g.standard_normal((H, W))
        W0 = g.standard_normal((H, W))
        Wt, Mt = W0.copy(), np.zeros((H, W))
        for _ in range(steps):
            Wt, Mt, _U = oracle.himuon_step(Wt, Mt, G, T, lr=lr, beta=beta, weight_decay=lam, nesterov=nesterov,
                                            scale_c=sc, lib=lib, **STEP)
        big = max(H, W)
        full = T == 0 or T >= big
        U = svd_closed_form(G, STEP["K"]) if full else _tilewise_closed_form(G, T, STEP["K"])
        tau = sc * np.sqrt(big if full else T)
        d = 1.0 - lr * lam
        W_ref = d ** steps * W0 - lr * tau * U * (1.0 - d ** steps) / (1.0 - d)
        M_ref = G * (1.0 - beta ** steps) / (1.0 - beta)
        worst = max(worst, rel(Wt, W_ref), rel(Mt, M_ref))
    return worst


def pin_step_nesterov_sign(lib=None):
    """Gradients G then -0.85 G with β = 0.9 from M = 0: the second direction
    is G (-0.85 + β² - 0.85 β) = -0.805 G with Nesterov (U = -Φ_K(G)) and the
    new buffer (β - 0.85) G = 0.05 G without it (U = +Φ_K(G))."""
    g = np.random.default_rng(22)
    G = g.standard_normal((40, 72))
    U_ref = svd_closed_form(G, STEP["K"])
    worst = 0.0
    for nesterov, sign in [(True, -1.0), (False, 1.0)]:
        Wt, Mt = np.zeros_like(G), np.zeros_like(G)
        Wt, Mt, U1 = oracle.himuon_step(Wt, Mt, G, 0, lr=0.1, beta=0.9, weight_decay=0.0, nesterov=nesterov,
                                        scale_c=0.2, lib=lib, **STEP)
        Wt, Mt, U2 = oracle.himuon_step(Wt, Mt, -0.85 * G, 0, lr=0.1, beta=0.9, weight_decay=0.0,
                                        nesterov=nesterov, scale_c=0.2, lib=lib, **STEP)
        tau = 0.2 * np.sqrt(72)
        worst = max(worst, rel(U1, U_ref), rel(U2, sign * U_ref), rel(Mt, 0.05 * G),
                    rel(Wt, -0.1 * tau * (1.0 + sign) * U_ref) if sign > 0 else rel(Wt, np.zeros_like(G)))
    return worst


def pin_step_scale_branch(lib=None):
    """Eq. (scaled_update): with W = 0, β = 0, λ = 0 one step leaves
    W = -lr τ U. T >= max(H, W) is the full map with τ = c sqrt(max(H, W));
    T < max(H, W) tiles with τ = c sqrt(T), also when T exceeds min(H, W)."""
    g = np.random.default_rng(23)
    worst = 0.0
    for (H, W, T) in [(48, 100, 64), (100, 48, 64), (48, 100, 100), (48, 100, 256), (100, 48, 0)]:
        G = g.standard_normal((H, W))
        Wt, _M, U = oracle.himuon_step(np.zeros((H, W)), np.zeros((H, W)), G, T, lr=0.5, beta=0.0,
                                       weight_decay=0.0, nesterov=False, scale_c=0.2, lib=lib, **STEP)
        full = T == 0 or T >= max(H, W)
        U_ref = svd_closed_form(G, STEP["K"]) if full else _tilewise_closed_form(G, T, STEP["K"])
        tau = 0.2 * np.sqrt(max(H, W) if full else T)
        worst = max(worst, rel(U, U_ref), rel(Wt, -0.5 * tau * U_ref))
    return worst


PINS = [
    pin_svd_closed_form, pin_tiled_blocks, pin_sampled_tiles, pin_rank_one, pin_scaled_orthogonal,
    pin_diagonal, pin_zero, pin_special_coefficients, pin_cubic_polar, pin_invariances,
    pin_tile_permutation, pin_single_tile_is_full_map, pin_tile_count,
    pin_step_constant_gradient, pin_step_nesterov_sign, pin_step_scale_branch, pin_rect_tiled_blocks,
]


def run_all(lib_path=None) -> int:
    """Run every pin; print each result; return the number that failed."""
    lib = oracle.load(lib_path) if lib_path else None
    failed = 0
    for pin in PINS:
        try:
            e = pin(lib)
            ok = bool(np.isfinite(e)) and e <= TOL
        except Exception as exc:  # a mutant may also raise
            e, ok = repr(exc), False
        failed += not ok
        print(f"{pin.__name__}: {'ok' if ok else 'FAIL'} ({e})", flush=True)
    return failed


if __name__ == "__main__":
    sys.exit(1 if run_all(sys.argv[1] if len(sys.argv) > 1 else None) else 0)
