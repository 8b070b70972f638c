"""Plain CPU oracle for the MuonBP optimizer step (fp64 numpy).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call
this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, constants
generator or helper with the HIP library; both sides only consume the same
seeded inputs from ``paper_2510_16981_amd.workload``.

Source: Khaled et al., "MuonBP: Faster Muon via Block-Periodic
Orthogonalization" (arXiv 2510.16981).

* ``orthogonalize_via_ns``   -- Algorithm 2 (Appendix B, Orthogonalize-via-NS).
* ``is_full_step``           -- the ``t mod P = 0`` test of Algorithm 1 (Sec. 3.2).
* ``block_ranges``           -- the r x c shard grid of Sec. 3 ("How blocks align
                                with model-parallel shards").
* ``orthogonalize_blockwise``-- BlockMuon's per-shard orthogonalization (Sec. 3.1).
* ``MuonBPOracle.step``      -- one iteration of Algorithm 1 (Sec. 3.2), with the
                                decoupled weight decay of Appendix B and the
                                optional RMS-matching scale of Sec. 3.2
                                ("AdamW learning rate transfer").
* ``ns_dense_flops``         -- the per-matrix cost model of Sec. 2.2
                                ("Computational costs") and its blockwise form
                                in Sec. 3 (first bullet).

Readings taken where the paper is silent (each is listed with its reason in
the design notes of the repository):

* the norm in Algorithm 2's normalisation is the Frobenius norm, and epsilon
  is added to the norm (not to its square);
* when a matrix has more rows than columns, NS runs on its transpose and the
  result is transposed back (the cost model of Sec. 2.2 assumes m <= n
  "without loss of generality"); in exact arithmetic both orders agree;
* period ``P = 0`` encodes P = infinity (BlockMuon): no step is full,
  including t = 0;  for finite P, t = 0 is a full step;
* weight decay is decoupled and scaled by the current step's learning rate:
  X <- X - eta_t (lambda X + s U);
* RMS matching multiplies U by beta * sqrt(max(p, q)) where p x q is the shape
  of the orthogonalized unit (block on block steps, matrix on full steps);
* Nesterov momentum (NS input G + mu M, M after this step's update) is an
  option that the paper does not state;  it is off by default, and its input
  is pinned by closed forms over two steps (tests of the oracle).

Every function here works in float64 on the exact values it is given.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Sequence, Tuple

import numpy as np

# Algorithm 2 fixes the quintic coefficients and epsilon.
NS_A, NS_B, NS_C = 2.0, -1.5, 0.5
NS_EPS = 1e-7


def ns_coefficients(coeffs, K: int) -> List[Tuple[float, float, float]]:
    """(a, b, c) of each of the K iterations.  ``coeffs`` is one triple (the
    same quintic every iteration, as printed in Algorithm 2) or a table of
    triples, one per iteration, whose last entry repeats past its end (the
    tuned or per-iteration coefficients that Sec. 2.2 mentions)."""
    arr = np.asarray(coeffs, dtype=np.float64)
    if arr.ndim == 1:
        if arr.shape != (3,):
            raise ValueError("coeffs must be (a, b, c) or a table of them")
        return [tuple(arr)] * K
    if arr.ndim != 2 or arr.shape[1] != 3 or arr.shape[0] == 0:
        raise ValueError("coeffs must be (a, b, c) or a table of them")
    return [tuple(arr[min(k, arr.shape[0] - 1)]) for k in range(K)]


def orthogonalize_via_ns(G, K: int = 5, eps: float = NS_EPS,
                         coeffs=(NS_A, NS_B, NS_C),
                         transpose_tall: bool = True) -> np.ndarray:
    """Algorithm 2 (Orthogonalize-via-NS), in fp64.

    The input is scaled to unit Frobenius norm (plus eps), which puts every
    singular value in [0, 1].  Each of the K iterations then maps every
    singular value x to the odd quintic p_k(x) = a_k x + b_k x^3 + c_k x^5
    and keeps the singular vectors.  As a matrix function on the left Gram
    matrix, whose eigenvalues are the squared singular values, that is
    X <- q_k(X X^T) X with q_k(lam) = a_k + b_k lam + c_k lam^2, evaluated
    here in Horner form.  Iteration k's (a_k, b_k, c_k) come from
    ``ns_coefficients``.  With ``transpose_tall`` the iteration runs on G^T
    when G has more rows than columns and the result is transposed back
    (the same matrix function, on the smaller Gram matrix).
    """
    table = ns_coefficients(coeffs, K)
    G = np.asarray(G, dtype=np.float64)
    if G.ndim != 2:
        raise ValueError("G must be a matrix")
    transposed = transpose_tall and G.shape[0] > G.shape[1]
    if transposed:
        G = G.T
    X = G / (np.linalg.norm(G, "fro") + eps)
    eye = np.eye(X.shape[0])
    for a, b, c in table:
        gram = X @ X.T
        q = a * eye + gram @ (b * eye + c * gram)  # q_k(X X^T)
        X = q @ X
    return X.T.copy() if transposed else X


def is_full_step(t: int, period: int) -> bool:
    """Algorithm 1's branch: full orthogonalization iff t mod P = 0.

    ``period == 0`` stands for P = infinity (BlockMuon, Sec. 3.1): never full.
    """
    if t < 0:
        raise ValueError("step must be >= 0")
    if period < 0:
        raise ValueError("period must be >= 0")
    return period > 0 and t % period == 0


def block_ranges(m: int, n: int, r: int, c: int) -> List[Tuple[slice, slice]]:
    """Shard grid of Sec. 3: W (m x n) cut into r x c blocks of m/r x n/c.

    Block (i, j) holds rows [i m/r, (i+1) m/r) and columns [j n/c, (j+1) n/c);
    the list is in row-major block order.
    """
    if r <= 0 or c <= 0 or m % r or n % c:
        raise ValueError("grid must divide the matrix evenly")
    mb, nb = m // r, n // c
    return [(slice(i * mb, (i + 1) * mb), slice(j * nb, (j + 1) * nb))
            for i in range(r) for j in range(c)]


def orthogonalize_blockwise(M, grid: Tuple[int, int], K: int = 5,
                            eps: float = NS_EPS,
                            coeffs=(NS_A, NS_B, NS_C)) -> np.ndarray:
    """BlockMuon's orthogonalization (Sec. 3.1): NS on every block alone."""
    M = np.asarray(M, dtype=np.float64)
    U = np.empty_like(M)
    for rs, cs in block_ranges(M.shape[0], M.shape[1], *grid):
        U[rs, cs] = orthogonalize_via_ns(M[rs, cs], K=K, eps=eps, coeffs=coeffs)
    return U


def momentum_update(M, G, mu: float) -> np.ndarray:
    """NTR momentum (eq. NTR, Algorithm 1): M_t = mu M_{t-1} + G_t."""
    return mu * np.asarray(M, dtype=np.float64) + np.asarray(G, dtype=np.float64)


def rms_scale(p: int, q: int, beta: float) -> float:
    """Sec. 3.2, AdamW learning-rate transfer: scale by beta * sqrt(max(p, q))."""
    return beta * math.sqrt(max(p, q))


def ns_dense_flops(m: int, n: int, K: int) -> float:
    """Cost of K NS iterations on an m x n matrix (Sec. 2.2): 2K(2 n m^2 + m^3)
    with m <= n; the momentum term 2mn is not included."""
    s, l = min(m, n), max(m, n)
    return 2.0 * K * (2.0 * l * s * s + s ** 3)


def ns_blockwise_dense_flops(m: int, n: int, r: int, c: int, K: int) -> float:
    """Same cost summed over the r x c blocks (Sec. 3, first bullet)."""
    return r * c * ns_dense_flops(m // r, n // c, K)


@dataclass
class MatrixSpec:
    rows: int
    cols: int
    grid_rows: int = 1
    grid_cols: int = 1


@dataclass
class OracleConfig:
    period: int = 5            # 0 = infinity
    lr_block: float = 0.02
    lr_full: float = 0.02
    momentum: float = 0.95
    weight_decay: float = 0.0
    ns_steps: int = 5
    eps: float = NS_EPS
    coeffs: tuple = (NS_A, NS_B, NS_C)  # one (a, b, c), or a per-iteration table
    nesterov: bool = False
    scale_mode: int = 0        # 0: s = 1 (Algorithm 1);  1: RMS matching
    rms_beta: float = 1.0


@dataclass
class StepRecord:
    full: bool
    M: List[np.ndarray] = field(default_factory=list)
    U: List[np.ndarray] = field(default_factory=list)


class MuonBPOracle:
    """Algorithm 1 (MuonBP) over a list of matrices, one CPU state per matrix.

    Momentum starts at zero (Algorithm 1, first line).  On a full step the
    whole matrix is orthogonalized ("gather" on a real cluster); otherwise
    every block of its grid is orthogonalized on its own.
    """

    def __init__(self, mats: Sequence[MatrixSpec], cfg: OracleConfig):
        self.mats = list(mats)
        self.cfg = cfg
        for s in self.mats:
            block_ranges(s.rows, s.cols, s.grid_rows, s.grid_cols)  # validate
        self.M = [np.zeros((s.rows, s.cols)) for s in self.mats]

    def orthogonalize(self, k: int, Y: np.ndarray, full: bool) -> np.ndarray:
        """U for matrix k: full NS, or NS per block, times the RMS scale."""
        cfg, spec = self.cfg, self.mats[k]
        ns = dict(K=cfg.ns_steps, eps=cfg.eps, coeffs=cfg.coeffs)
        if full:
            U = orthogonalize_via_ns(Y, **ns)
            if cfg.scale_mode == 1:
                U = U * rms_scale(spec.rows, spec.cols, cfg.rms_beta)
            return U
        U = orthogonalize_blockwise(Y, (spec.grid_rows, spec.grid_cols), **ns)
        if cfg.scale_mode == 1:
            U = U * rms_scale(spec.rows // spec.grid_rows,
                              spec.cols // spec.grid_cols, cfg.rms_beta)
        return U

    def step(self, params: List[np.ndarray], grads: List[np.ndarray], t: int,
             record: bool = False):
        """One iteration t of Algorithm 1.  Returns the new params (fp64)."""
        cfg = self.cfg
        full = is_full_step(t, cfg.period)
        eta = cfg.lr_full if full else cfg.lr_block
        rec = StepRecord(full=full)
        out = []
        for k, (X, G) in enumerate(zip(params, grads)):
            G = np.asarray(G, dtype=np.float64)
            X = np.asarray(X, dtype=np.float64)
            self.M[k] = momentum_update(self.M[k], G, cfg.momentum)
            Y = G + cfg.momentum * self.M[k] if cfg.nesterov else self.M[k]
            U = self.orthogonalize(k, Y, full)
            out.append(X - eta * (cfg.weight_decay * X + U))
            if record:
                rec.M.append(self.M[k].copy())
                rec.U.append(U)
        return (out, rec) if record else out
