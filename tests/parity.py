"""Per-tile comparison of the HIP path with the fp64 oracle.

The error measure is the per-tile relative Frobenius error
e = ||Y_gpu - Y_oracle||_F / ||Y_oracle||_F over the unpadded part of each
tile; a tile whose oracle output is exactly zero must come back exactly zero.
Bars: 1e-5 for fp32 storage, 2e-2 for bf16 storage.
"""
import numpy as np
import torch

TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}

# bf16 storage with bf16 MFMA operands (HIMUON_COMPUTE_BF16, opt-in only; the
# default for bf16 storage is fp16 operands, which meet the 2e-2 bar). A bf16
# operand keeps 8 significant bits (unit roundoff u = 2^-9), and each step
# rounds three product operands whose errors the map carries forward: one
# step amplifies small singular values by up to a = 3.44, and the step's
# cancellation (aX + BX with B near (1 - a)I) by about 2a. Measured worst
# tiles (config 2 and config 5 shapes): 1.2e-2 at T = 256, 2.1e-2 at
# T = 128, 2.9e-2 at T = 32 for K = 5; up to 6.9e-2 (35 u) at T = 32, K = 8.
# This mode is held to 64 u: a bar that catches a wrong term (an O(1) error)
# but not the format's own rounding. It does not meet the 2e-2 target at
# T <= 64 or K = 8.
BF16_OPERAND_BAR = 64 * 2.0 ** -9
COEF32 = tuple(float(np.float32(v)) for v in (3.4445, -4.7750, 2.0315))  # what the ABI receives


def to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact widening of the device values (fp32 or bf16) to float64."""
    return t.detach().float().cpu().double().numpy()


def tile_errors(Y, R, T):
    """Per-tile relative errors (row-major over the tile grid)."""
    Y = np.asarray(Y, dtype=np.float64)
    R = np.asarray(R, dtype=np.float64)
    H, W = R.shape
    out = []
    for r0 in range(0, H, T):
        for c0 in range(0, W, T):
            y = Y[r0:r0 + T, c0:c0 + T]
            r = R[r0:r0 + T, c0:c0 + T]
            nr = np.linalg.norm(r)
            if nr == 0.0:
                out.append(0.0 if not np.any(y) else np.inf)
            else:
                out.append(np.linalg.norm(y - r) / nr)
    return np.array(out)


def sampled_tile_errors(Y, tiles_orc, ids, T):
    """Errors for oracle tiles (each T x T, padded) at tile ids of matrix Y."""
    H, W = Y.shape
    C = -(-W // T)
    errs = []
    for s, t in enumerate(ids):
        r, c = divmod(int(t), C)
        y = np.asarray(Y[r * T:(r + 1) * T, c * T:(c + 1) * T], dtype=np.float64)
        ref = tiles_orc[s][:y.shape[0], :y.shape[1]]
        nr = np.linalg.norm(ref)
        errs.append((0.0 if not np.any(y) else np.inf) if nr == 0 else np.linalg.norm(y - ref) / nr)
    return np.array(errs)
