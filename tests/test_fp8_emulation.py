"""Why the map has no fp8e4m3-operand kernel: an emulation, checked on the CPU.

The paper's precision study (Sec. 6.5, Tab. precision_recovery) runs the
Newton-Schulz GEMMs with fp8e4m3 operands. Here that scheme is emulated on
single tiles: each step quantises the three product operands X, A = X X^T and
B = bA + cA^2 to e4m3 after a dynamic per-tile scale (largest magnitude to
448, e4m3's largest finite value), forms the products and the combinations
aX + BX, bA + cA^2 in fp64, and keeps an fp64 master iterate. The result is
compared, tile by tile, with the fp64 oracle (oracle.phi_k on the tile).

The e4m3 rounding is pinned first against the format itself: all 127
non-negative finite e4m3 values are decoded from their bit patterns (1 sign,
4 exponent bits with bias 7, 3 mantissa bits; subnormals at exponent field 0;
the all-ones pattern is NaN, there is no infinity), and the emulator must
return the nearest of them, ties to the even code, saturating at 448.

The emulator is calibrated with bf16 operands in place of e4m3: the bf16-
operand kernel measures 1.85e-2 on config 2 at T = 128, K = 5 on the GPU, and
the emulator must land in the same range. With e4m3 operands the per-tile
error is an order of magnitude above the 2e-2 bar of bf16 storage (at every
tile size the fused kernels serve and at T = 512), and still above it with
e4m3 in the Gram product alone. The step's cancellation is the cause: near
convergence B is close to (1 - a) I with a = 3.4445, so aX + BX subtracts two
terms about three times larger than the result, which amplifies e4m3's 2^-4
relative rounding of B. The completed-square form of the fp16 kernels
(aI + P = sigma M^2 + a' I as one operand) has no such cancellation, yet
with e4m3 operands it is still several times over the bar: the iterate itself
is rounded to e4m3 at every step. (The paper's 2-6% figures are operator gaps
of the diagnostic's one-step weights, not per-tile errors of the map.)
"""
import numpy as np
import pytest

import oracle

A_, B_, C_ = 3.4445, -4.7750, 2.0315
BF16_BAR = 2e-2


# ------------------------------------------------------------ e4m3 format

def e4m3_values():
    """All non-negative finite e4m3 values, decoded from codes 0x00..0x7E."""
    vals = []
    for code in range(0x7F):
        e, m = code >> 3, code & 7
        vals.append(m * 2.0 ** -9 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7))
    return np.array(vals)


def to_e4m3(x):
    """Round to nearest e4m3 (ties to even), saturating at 448: the exponent
    of the result's binade fixes a spacing of 2^(e-3), or 2^-9 below 2^-6."""
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -30)))
    q = 2.0 ** (np.maximum(e, -6.0) - 3.0)
    r = np.minimum(np.round(a / q) * q, 448.0)  # np.round: half to even
    return np.sign(x) * r


def test_e4m3_rounding_matches_the_format():
    vals = e4m3_values()
    assert len(np.unique(vals)) == 127 and vals.max() == 448.0 and vals[1] == 2.0 ** -9
    # every value is a fixed point
    assert np.array_equal(to_e4m3(vals), vals)
    # random magnitudes: nearest value, ties to the even code
    rng = np.random.default_rng(0)
    x = np.concatenate([np.exp(rng.uniform(np.log(2.0 ** -12), np.log(440.0), 20000)),
                        (vals[:-1] + vals[1:]) / 2])  # exact midpoints
    r = to_e4m3(x)
    for xi, ri in zip(x, r):
        d = np.abs(vals - xi)
        best = np.flatnonzero(d == d.min())
        want = vals[best[0]] if len(best) == 1 else vals[[b for b in best if b % 2 == 0][0]]
        assert ri == want, (xi, ri, want)
    assert to_e4m3(1000.0) == 448.0 and to_e4m3(-1000.0) == -448.0
    assert to_e4m3(-0.3) == -to_e4m3(0.3)


def to_bf16(x):
    """Round to bf16 (nearest even), through the fp32 bit pattern."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


# ------------------------------------------------------------ emulated map

def scaled(q, x):
    """x as q-rounded operand with a dynamic per-tile scale (amax -> 448 for
    e4m3; none for bf16, which has fp32's range): returns (operand, scale)."""
    if q is to_e4m3:
        amax = np.abs(x).max()
        s = amax / 448.0 if amax > 0 else 1.0
        return q(x / s), s
    return q(x), 1.0


def phi_quantised(S, K, q, gram_only=False):
    X = S / np.linalg.norm(S)
    for _ in range(K):
        Xq, sx = scaled(q, X)
        A = sx * sx * (Xq @ Xq.T)
        if gram_only:
            X = A_ * X + (B_ * A + C_ * (A @ A)) @ X
            continue
        Aq, sa = scaled(q, A)
        B = B_ * A + C_ * sa * sa * (Aq @ Aq.T)
        Bq, sb = scaled(q, B)
        X = A_ * X + sb * sx * (Bq @ Xq)
    return X


def tiles(kind, T, n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        if kind == "gaussian":
            out.append(rng.standard_normal((T, T)))
        else:  # low rank (16, sigma_i = 1/i) plus 0.01 N(0, 1)
            U, _ = np.linalg.qr(rng.standard_normal((T, 16)))
            V, _ = np.linalg.qr(rng.standard_normal((T, 16)))
            out.append(U @ np.diag(1.0 / np.arange(1, 17)) @ V.T + 0.01 * rng.standard_normal((T, T)))
    return out


def errors(kind, T, q, n=3, K=5, gram_only=False, seed=1):
    errs = []
    for S in tiles(kind, T, n, seed):
        R = oracle.phi_k(S, K, A_, B_, C_)
        Y = phi_quantised(S, K, q, gram_only)
        errs.append(np.linalg.norm(Y - R) / np.linalg.norm(R))
    return np.array(errs)


def test_emulator_calibrated_by_bf16_operands():
    """bf16 in place of e4m3: the emulator lands where the bf16-operand
    kernel does (1.85e-2 at T = 128, K = 5 on the GPU), just under the bar."""
    e = errors("gaussian", 128, to_bf16, n=4)
    print(f"bf16 operands, T=128: {e}")
    assert 1.0e-2 <= e.max() <= 2.5e-2


@pytest.mark.parametrize("T", [64, 128, 256, 512])
@pytest.mark.parametrize("kind", ["gaussian", "lowrank"])
def test_fp8_operands_miss_the_bf16_bar(T, kind):
    e = errors(kind, T, to_e4m3, n=2 if T == 512 else 3)
    print(f"e4m3 operands, {kind}, T={T}: {e}")
    # every tile is at least five times over the 2e-2 bar
    assert e.min() >= 5 * BF16_BAR


def phi_quantised_completed(S, K, q):
    """The step in the form the fp16 kernels use (rescaled state Z = X
    |c|^(1/4), M = Z Z^T + (sigma b'/2) I from the Gram accumulator, aI + P =
    sigma M^2 + a' I with a' = a - b^2 / (4c), Z <- (aI + P) Z), every product
    operand (Z, M, aI + P) q-rounded after its per-tile scale."""
    T = S.shape[0]
    zs = abs(C_) ** 0.25
    bq = B_ / np.sqrt(abs(C_))
    am = A_ - B_ * B_ / (4 * C_)
    Z = S * (zs / np.linalg.norm(S))
    eye = np.eye(T)
    for _ in range(K):
        Zq, sz = scaled(q, Z)
        M = sz * sz * (Zq @ Zq.T) + (bq / 2) * eye
        Mq, sm = scaled(q, M)
        P = sm * sm * (Mq @ Mq) + am * eye
        Pq, sp = scaled(q, P)
        Z = sp * sz * (Pq @ Zq)
    return Z / zs


@pytest.mark.parametrize("T", [128, 256])
def test_fp8_misses_the_bar_in_the_completed_square_form_too(T):
    """The completed square removes the cancellation of aI against BX, and
    bf16 operands then land at about 1.2e-2; e4m3 operands still leave every
    tile several times over the bar, the e4m3 rounding of the iterate itself
    (2^-4 relative, at every step) being the cause."""
    errs = {}
    for name, q in (("bf16", to_bf16), ("e4m3", to_e4m3)):
        e = []
        for S in tiles("lowrank", T, 2, 1):
            R = oracle.phi_k(S, 5, A_, B_, C_)
            e.append(np.linalg.norm(phi_quantised_completed(S, 5, q) - R) / np.linalg.norm(R))
        errs[name] = np.array(e)
        print(f"{name} operands, completed square, T={T}: {errs[name]}")
    assert errs["bf16"].max() <= BF16_BAR
    assert errs["e4m3"].min() >= 5 * BF16_BAR


@pytest.mark.parametrize("T", [128, 256])
def test_fp8_in_the_gram_product_alone_misses_the_bar(T):
    e = errors("gaussian", T, to_e4m3, gram_only=True)
    print(f"e4m3 Gram only, T={T}: {e}")
    assert e.min() >= 2 * BF16_BAR
