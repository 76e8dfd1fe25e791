"""Seeded input generators (numpy PCG64) with the shapes and value
distributions of the workloads the layer is measured on.

Recipe (one LC-VQ weight matrix, index k within a workload):
  * map A (d x d, fp32)  = 0.02 * (I + 0.1 * N(0,1)),      seed 1000 + k
  * offset b (d, fp32)   = 0.005 * N(0,1),                  seed 2000 + k
  * latent Z (m x n)     ~ U(lo, hi), default U(-0.5, 3.5), seed 3000 + k
  * activations X (N x n) ~ N(0,1),                          seed 4000 + k
  * upstream grad dY (N x m) ~ N(0,1),                       seed 5000 + k
Values are drawn in fp32; bf16 tensors are the round-to-nearest-even cast of
those fp32 draws, done once here, so every consumer sees the same bits.
"""
from __future__ import annotations

import numpy as np

# Llama-shaped layers: (name, [(m, n), ...], N tokens, dtype).  Z, X and dY
# are bf16 except in the small fp32 case.
WORKLOADS = {
    "lcvq_256x256_n16_fp32": dict(mats=[(256, 256)], N=16, dtype="f32", d=8),
    "lcvq_4096x4096_n4096_bf16": dict(mats=[(4096, 4096)], N=4096, dtype="bf16", d=8),
    "lcvq_mlp7b_n8192_bf16": dict(mats=[(11008, 4096), (11008, 4096), (4096, 11008)], N=8192,
                                  dtype="bf16", d=8),
    "lcvq_mlp70b_n4096_bf16": dict(mats=[(28672, 8192), (8192, 28672)], N=4096, dtype="bf16", d=8),
    "lcvq_block7b_n16384_bf16": dict(mats=[(4096, 4096)] * 4 + [(11008, 4096), (11008, 4096), (4096, 11008)],
                                     N=16384, dtype="bf16", d=8),
}


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def bf16_bits(x) -> np.ndarray:
    """fp32 -> bf16 storage bits (uint16), round to nearest even; NaN stays a quiet NaN."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(f)
    out = np.where(nan, (u >> 16) | 0x40, rounded).astype(np.uint16)
    return out


def bf16_bits_to_f32(bits) -> np.ndarray:
    """Exact widening of bf16 storage bits to fp32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def draw_map(d: int, k: int = 0):
    """(A, b) in fp32 with the recipe above."""
    A = (0.02 * (np.eye(d) + 0.1 * rng(1000 + k).standard_normal((d, d)))).astype(np.float32)
    b = (0.005 * rng(2000 + k).standard_normal(d)).astype(np.float32)
    return A, b


def _store(x32: np.ndarray, dtype: str):
    if dtype == "f32":
        return x32
    if dtype == "bf16":
        return bf16_bits(x32)
    raise ValueError(dtype)


def draw_latent(m: int, n: int, k: int = 0, dtype: str = "bf16", lo: float = -0.5, hi: float = 3.5):
    z = rng(3000 + k).uniform(lo, hi, size=(m, n)).astype(np.float32)
    return _store(z, dtype)


def draw_activations(rows: int, cols: int, seed: int, dtype: str = "bf16"):
    x = rng(seed).standard_normal((rows, cols), dtype=np.float32)
    return _store(x, dtype)


def layer_inputs(N: int, m: int, n: int, d: int, dtype: str = "bf16", k: int = 0,
                 z_lo: float = -0.5, z_hi: float = 3.5) -> dict:
    """All inputs of one fwd+bwd call in storage form: fp32 arrays, or uint16
    bf16 bits when dtype == 'bf16'.  A and b are always fp32."""
    A, b = draw_map(d, k)
    return dict(
        N=N, m=m, n=n, d=d, dtype=dtype,
        A=A, b=b,
        Z=draw_latent(m, n, k, dtype, z_lo, z_hi),
        X=draw_activations(N, n, 4000 + k, dtype),
        dY=draw_activations(N, m, 5000 + k, dtype),
    )
