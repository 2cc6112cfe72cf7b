"""The fp32-operand kernels normalise a tile by a power of two only and carry
the rest of its norm in the step's coefficients; checked here on the CPU.

A step of the quintic iteration (Sec. 2.2, eqs. ns_iteration / ns_quintic) is
homogeneous: with X = Y / rho,
    aX + (bA + cA^2) X = (aY + ((b/rho^2) A_Y + (c/rho^4) A_Y^2) Y) / rho,
A = X X^T, A_Y = Y Y^T. Phi_K (eq. phi_k_def) starts from X_0 = S / ||S||_F;
taking Y_0 = S 2^-e with ||Y_0||_F^2 = m in [1, 4) and rho = sqrt(m), the
iteration on Y with coefficients (a, b/m, c/m^2) ends at Y_K = rho X_K. In
fp32 the power-of-two scale is exact, so the normalised tile is never
rounded. These tests check the identity in fp64 against the oracle, and
evaluate both forms with fp32 products (numpy) on heavy-tailed tiles at
K = 8, where the per-tile errors of either form reach to just under the
1e-5 bar. This is test infrastructure only; the GPU parity tests check the
kernels.
"""
import numpy as np
import pytest

import oracle
import workloads
from parity import COEF32

A, B, C = COEF32


def split_norm(S):
    """(Y_0, m): S 2^-e with ||Y_0||_F^2 = m in [1, 4)."""
    ss = float((S * S).sum())
    e = int(np.floor(np.log2(ss) / 2))
    Y = S * 2.0 ** -e
    m = float((Y * Y).sum())
    if m >= 4.0:  # log2 rounding at a power of four
        Y, m = Y / 2, m / 4
    return Y, m


def fma(a, b, c, dt):
    """a b + c rounded once to dt (the fp64 product of two fp32 numbers is exact)."""
    return (np.float64(a) * np.asarray(b, np.float64) + np.asarray(c, np.float64)).astype(dt)


def phi_y(S, K, dt):
    """The kernels' form: Y_0 = S 2^-e, coefficients b/m and c/m^2 as
    hi + lo pairs, B = fma(ch, A^2, fma(bh, A, fma(bl, A, cl A^2)))."""
    Y, m = split_norm(S)
    bd, cd = B / m, C / (m * m)
    bh, ch = dt(bd), dt(cd)
    bl, cl = dt(bd - np.float64(bh)), dt(cd - np.float64(ch))
    Y = Y.astype(dt)
    for _ in range(K):
        G = (Y @ Y.T).astype(dt)
        Q = (G @ G).astype(dt)
        t = fma(bl, G, (cl * Q).astype(dt), dt)
        Bm = fma(ch, Q, fma(bh, G, t, dt), dt)
        Y = fma(A, Y, (Bm @ Y).astype(dt), dt)
    return Y.astype(np.float64) * dt(1.0 / np.sqrt(m))


def phi_x(S, K, dt):
    """The earlier form: X_0 = S / ||S||_F rounded, B = fma(c, A^2, b A)."""
    X = (S / np.linalg.norm(S)).astype(dt)
    for _ in range(K):
        G = (X @ X.T).astype(dt)
        Q = (G @ G).astype(dt)
        Bm = fma(C, Q, (dt(B) * G).astype(dt), dt)
        X = fma(A, X, (Bm @ X).astype(dt), dt)
    return X.astype(np.float64)


def test_split_norm_is_exact_and_in_range():
    rng = np.random.default_rng(3)
    for scale in (1e-30, 1e-3, 1.0, 7.0, 1e20):
        S = scale * rng.standard_normal((32, 48))
        Y, m = split_norm(S)
        assert 1.0 <= m < 4.0
        ratio = S / Y
        assert np.all(ratio == ratio.flat[0])  # one power of two for every entry
        assert np.log2(ratio.flat[0]) == np.round(np.log2(ratio.flat[0]))


@pytest.mark.parametrize("shape,K", [((32, 32), 5), ((64, 48), 8), ((48, 64), 3)])
def test_identity_in_fp64(shape, K):
    S = workloads.student_t(*shape, 77, "f32").numpy().astype(np.float64)
    R = oracle.phi_k(S, K, A, B, C)
    Y = phi_y(S, K, np.float64)
    assert np.linalg.norm(Y - R) / np.linalg.norm(R) < 1e-12


def test_fp32_floor_of_the_map_on_heavy_tailed_tiles():
    """Heavy-tailed 32-tiles at K = 8 (the fp32 path's hardest case), 1024
    tiles, both forms evaluated with fp32 products: the median per-tile error
    is the same (about 1.4e-6) and the largest tiles sit just under the 1e-5
    bar in both, so that bar is close to what fp32 arithmetic allows for this
    map at K = 8, whichever form; which tile is worst is a matter of rounding
    luck. Removing the rounding of X_0 takes one error source away without
    adding another."""
    x = workloads.student_t(1024, 1024, 5017, "f32").numpy().astype(np.float64)
    ex, ey = [], []
    for r in range(0, 1024, 32):
        for c in range(0, 1024, 32):
            S = x[r:r + 32, c:c + 32]
            R = oracle.phi_k(S, 8, A, B, C)
            n = np.linalg.norm(R)
            ex.append(np.linalg.norm(phi_x(S, 8, np.float32) - R) / n)
            ey.append(np.linalg.norm(phi_y(S, 8, np.float32) - R) / n)
    ex, ey = np.array(ex), np.array(ey)
    p99x, p99y = np.percentile(ex, 99), np.percentile(ey, 99)
    print(f"fp32, rounded X_0: max {ex.max():.3e} p99 {p99x:.3e} p50 {np.median(ex):.3e}; "
          f"exact scale: max {ey.max():.3e} p99 {p99y:.3e} p50 {np.median(ey):.3e}")
    assert abs(np.median(ey) / np.median(ex) - 1) < 0.03
    assert 0.5e-5 < ex.max() < 1e-5 and 0.5e-5 < ey.max() < 1e-5
