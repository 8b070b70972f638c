"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module draws matrices and casts them; it performs none of the optimizer's
arithmetic.  Both the CPU oracle and the HIP path consume exactly the values it
returns (the oracle widens them to float64).

Gradient model (a stand-in for the paper's language-model workloads, whose data
and weights are not available): for matrix k,

    G_t = U diag(s) V^T + E_t,   s_i = 1 / i (i = 1..rank),
    U, V = orthonormal bases from QR of standard normal matrices,
    E_t ~ N(0, noise_std^2) elementwise (noise_std = 1e-3),

and initial weights X_0 ~ N(0, 0.02^2).  Every draw has its own
``numpy.random.default_rng`` stream keyed by (seed, kind, k[, t]) so that any
matrix or step can be regenerated alone.
"""

from __future__ import annotations

import numpy as np

_KIND_BASIS, _KIND_NOISE, _KIND_PARAM = 0, 1, 2

# Shapes: W is rows x cols (in x out, row-major); grid = (grid_rows, grid_cols).
# qkv-2048x6144: one fused attention QKV weight, 8-way column (TP) shards.
# dense-16L-d2048: 16 layers of a d=2048, ffn=8192 transformer, every matrix
#   8-way column-sharded.
# llama-32L-d4096: 32 layers of an 8B Llama-style model (d=4096, ffn=14336,
#   GQA kv width 1024), Megatron layout: column-parallel q, k, v, gate, up
#   (grid 1x8), row-parallel o and down (grid 8x1).
WORKLOADS = {
    "single-256x512-f32": dict(
        mats=[(256, 512, 1, 2)], dtype="f32", rank=32, period=5, steps=10),
    "qkv-2048x6144-bf16": dict(
        mats=[(2048, 6144, 1, 8)], dtype="bf16", rank=128, period=5, steps=100),
    "dense-16L-d2048-bf16": dict(
        mats=[(2048, 2048, 1, 8)] * 4 + [(2048, 8192, 1, 8)] * 2
        + [(8192, 2048, 1, 8)], layers=16, dtype="bf16", rank=128, period=5,
        steps=25),
    "llama-32L-d4096-bf16": dict(
        mats=[(4096, 4096, 1, 8), (4096, 1024, 1, 8), (4096, 1024, 1, 8),
              (4096, 4096, 8, 1), (4096, 14336, 1, 8), (4096, 14336, 1, 8),
              (14336, 4096, 8, 1)], layers=32, dtype="bf16", rank=128,
        period=5, steps=10),
    "mlp-4096x14336-full-and-4x2-bf16": dict(
        mats=[(4096, 14336, 4, 2), (14336, 4096, 4, 2)], dtype="bf16",
        rank=128, period=5, steps=10),
}

# Periods swept for the 8B-shaped model (P = 0 stands for infinity).
PERIOD_SWEEP = [1, 2, 5, 10, 0]


def workload_matrices(name: str):
    """List of (rows, cols, grid_rows, grid_cols) for a named workload."""
    w = WORKLOADS[name]
    return list(w["mats"]) * int(w.get("layers", 1))


def _rng(*key):
    return np.random.default_rng([int(v) for v in key])


def lowrank_basis(m: int, n: int, rank: int, seed: int, k: int):
    """Orthonormal U (m x r), V (n x r) and s_i = 1/i for matrix k."""
    r = min(rank, m, n)
    g = _rng(seed, _KIND_BASIS, k)
    U, _ = np.linalg.qr(g.standard_normal((m, r)))
    V, _ = np.linalg.qr(g.standard_normal((n, r)))
    s = 1.0 / np.arange(1, r + 1, dtype=np.float64)
    return U, s, V


def lowrank_grad(m: int, n: int, rank: int, seed: int, k: int, t: int,
                 noise_std: float = 1e-3, basis=None) -> np.ndarray:
    """G_t for matrix k (float64): U diag(s) V^T + N(0, noise_std^2) noise."""
    U, s, V = basis if basis is not None else lowrank_basis(m, n, rank, seed, k)
    G = (U * s) @ V.T
    G += noise_std * _rng(seed, _KIND_NOISE, k, t).standard_normal((m, n))
    return G


def init_param(m: int, n: int, seed: int, k: int, std: float = 0.02) -> np.ndarray:
    """X_0 for matrix k (float64), N(0, std^2)."""
    return std * _rng(seed, _KIND_PARAM, k).standard_normal((m, n))


def device_grad(m: int, n: int, rank: int, seed: int, k: int, noise_std: float = 1e-3,
                device: str = "cuda"):
    """Timing-only stand-in for lowrank_grad at model scale, drawn on the GPU
    (torch): a rank-`rank` product with singular values close to 1/i (the
    factors are Gaussian with columns scaled to unit expected norm, not
    orthonormalised) plus N(0, noise_std^2) noise, returned as bf16.  Its
    values differ from lowrank_grad's; use it only where nothing is checked
    against the oracle."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000003 + int(k))
    r = min(rank, m, n)
    U = torch.randn(m, r, generator=g, device=device) / m ** 0.5
    V = torch.randn(n, r, generator=g, device=device) / n ** 0.5
    s = 1.0 / torch.arange(1, r + 1, device=device, dtype=torch.float32)
    G = (U * s) @ V.T
    G += noise_std * torch.randn(m, n, generator=g, device=device)
    return G.to(torch.bfloat16)


def device_param(m: int, n: int, seed: int, k: int, std: float = 0.02, device: str = "cuda"):
    """Timing-only X_0 ~ N(0, std^2) drawn on the GPU, bf16."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000003 + int(k) + 7919)
    return (std * torch.randn(m, n, generator=g, device=device)).to(torch.bfloat16)


def quantize(x: np.ndarray, dtype: str):
    """Round a float64 array to the storage dtype ('f32' or 'bf16', RNE).

    Returns a CPU torch tensor; ``.double().numpy()`` gives the exact values
    the oracle must see.
    """
    import torch
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64)).to(tdt)
