"""Seeded synthetic inputs for the tiled Newton–Schulz map.

This module only draws random matrices. It holds none of the method's
arithmetic (no normalisation, no Newton–Schulz step, no tiling), so that the
fp64 oracle and the HIP path can both be fed from it without sharing any code
that decides a result.

Workloads (shapes and distributions are synthetic stand-ins; the paper's
training data, datasets and model weights are not used):

* ``gaussian``            i.i.d. N(0, 1) entries.
* ``lowrank_plus_noise``  a momentum-like matrix U·diag(σ)·Vᵀ + 0.01·N(0, 1)
                          with U, V orthonormal of rank 64 and σ_i = 1/i.
* ``student_t``           heavy-tailed 0.02·t(ν=3) entries.
* ``LAYER_7B``            the seven projection shapes of one 7B-style
                          transformer layer (q, k, v, o 4096×4096; gate, up
                          11008×4096; down 4096×11008).
* ``HETERO_SHAPES``       8 each of 1024×4096, 4096×1024 and 2048×2048.

Every generator is seeded; the low-rank factors come from numpy's PCG64 and
QR, the dense noise from a seeded ``torch.Generator`` on the target device
(so the 6.5e9-entry 32-layer stack can be drawn on the GPU in seconds).
Parity never depends on the generator being bit-portable: tests always hand
the oracle the exact bytes that sit in device memory.
"""
from __future__ import annotations

import numpy as np
import torch

QUINTIC = (3.4445, -4.7750, 2.0315)  # Muon's quintic coefficients, eq. (ns_quintic)

LAYER_7B = (
    ("q_proj", 4096, 4096),
    ("k_proj", 4096, 4096),
    ("v_proj", 4096, 4096),
    ("o_proj", 4096, 4096),
    ("gate_proj", 11008, 4096),
    ("up_proj", 11008, 4096),
    ("down_proj", 4096, 11008),
)

HETERO_SHAPES = tuple([(1024, 4096)] * 8 + [(4096, 1024)] * 8 + [(2048, 2048)] * 8)

# The seven Muon-eligible matrices of one transformer block of each Qwen3
# model, output x input (Sec. 6.3, Tab. qwen3_shapes), for the per-layer
# tiled/full comparison; the inputs themselves are random Gaussian.
QWEN3_BLOCK0 = {
    "0.6B": (("q_proj", 2048, 1024), ("k_proj", 1024, 1024), ("v_proj", 1024, 1024), ("o_proj", 1024, 2048),
             ("gate_proj", 3072, 1024), ("up_proj", 3072, 1024), ("down_proj", 1024, 3072)),
    "1.7B": (("q_proj", 2048, 2048), ("k_proj", 1024, 2048), ("v_proj", 1024, 2048), ("o_proj", 2048, 2048),
             ("gate_proj", 6144, 2048), ("up_proj", 6144, 2048), ("down_proj", 2048, 6144)),
    "4B": (("q_proj", 4096, 2560), ("k_proj", 1024, 2560), ("v_proj", 1024, 2560), ("o_proj", 2560, 4096),
           ("gate_proj", 9728, 2560), ("up_proj", 9728, 2560), ("down_proj", 2560, 9728)),
}

_TORCH_DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16, "f64": torch.float64}


def _cast(x: torch.Tensor, dtype: str) -> torch.Tensor:
    # torch's float32 -> bfloat16 conversion rounds to nearest even.
    return x.to(_TORCH_DTYPES[dtype]).contiguous()


def gaussian(H: int, W: int, seed: int, dtype: str = "f32", device="cpu") -> torch.Tensor:
    """i.i.d. N(0,1) drawn in fp64 by numpy's PCG64 stream ``default_rng(seed)``."""
    x = np.random.default_rng(seed).standard_normal((H, W))
    return _cast(torch.from_numpy(x).to(device), dtype)


def student_t(H: int, W: int, seed: int, dtype: str = "f32", device="cpu",
              scale: float = 0.02, nu: float = 3.0) -> torch.Tensor:
    """scale · t(ν) entries from ``default_rng(seed).standard_t``."""
    x = scale * np.random.default_rng(seed).standard_t(nu, size=(H, W))
    return _cast(torch.from_numpy(x).to(device), dtype)


def lowrank_plus_noise(H: int, W: int, seed: int, dtype: str = "bf16", device="cpu",
                       rank: int = 64, noise: float = 0.01) -> torch.Tensor:
    """U·diag(1/i)·Vᵀ + noise·N(0,1), U (H×rank) and V (W×rank) orthonormal.

    U and V are the Q factors of ``default_rng(seed)`` Gaussian draws; the
    dense noise comes from ``torch.Generator(device).manual_seed(seed)``.
    The sum is formed in fp32 and rounded once to ``dtype``.
    """
    rng = np.random.default_rng(seed)
    U, _ = np.linalg.qr(rng.standard_normal((H, rank)))
    V, _ = np.linalg.qr(rng.standard_normal((W, rank)))
    sig = 1.0 / np.arange(1, rank + 1, dtype=np.float64)
    Us = torch.from_numpy((U * sig).astype(np.float32)).to(device)
    Vt = torch.from_numpy(np.ascontiguousarray(V.T).astype(np.float32)).to(device)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    x = torch.randn((H, W), generator=gen, device=device, dtype=torch.float32)
    x.mul_(noise)
    x.addmm_(Us, Vt)
    return _cast(x, dtype)


def layer_7b(seed_base: int, dtype: str = "bf16", device="cpu"):
    """One 7B-style layer: seven low-rank-plus-noise matrices, seeds seed_base + j."""
    return [lowrank_plus_noise(H, W, seed_base + j, dtype, device)
            for j, (_, H, W) in enumerate(LAYER_7B)]


def stack_7b(n_layers: int = 32, dtype: str = "bf16", device="cpu", seed_base: int = 4000):
    """``n_layers`` copies of the 7B layer shapes, seeds seed_base + 7·L + j."""
    out = []
    for L in range(n_layers):
        out.extend(layer_7b(seed_base + 7 * L, dtype, device))
    return out


def heterogeneous(dtype: str = "f32", device="cpu", seed_base: int = 5000):
    """24 heavy-tailed matrices (8 each of three shapes), seeds seed_base + i."""
    return [student_t(H, W, seed_base + i, dtype, device)
            for i, (H, W) in enumerate(HETERO_SHAPES)]


def stack_7b_shapes(n_layers: int = 32):
    return [(H, W) for _ in range(n_layers) for (_, H, W) in LAYER_7B]
