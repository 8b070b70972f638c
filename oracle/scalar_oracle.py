"""Plain CPU oracle for the optimizer pieces around MuonBP (fp64 numpy).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call
this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library.

The paper trains the parameters MuonBP does not orthogonalize (1D parameters
and the input embedding) with AdamW, clips their gradients to a global norm of
1.0, uses weight decay 0.1, and schedules the learning rate with cosine decay
(960M / 1.2B runs) or warmup-stable-decay with a linear decay to a final value
(8B runs; no warmup and a 20% cooldown in the 160M comparison).  Appendix B
(experimental details) and Sec. 4 (experiments) state these choices.

* ``clip_factor``  -- global-norm gradient clipping: every gradient is scaled
                      by min(1, max_norm / (||g||_2 + 1e-6)), ||g||_2 over all
                      the tensors together; max_norm = 0 turns it off.
* ``adamw_step``   -- one AdamW iteration (Adam's moments with bias correction,
                      Kingma & Ba; decoupled weight decay, Loshchilov & Hutter):
                          p <- p (1 - lr wd)
                          m <- b1 m + (1 - b1) g,  v <- b2 v + (1 - b2) g^2
                          p <- p - lr m_hat / (sqrt(v_hat) + eps),
                      m_hat = m / (1 - b1^t), v_hat = v / (1 - b2^t), t = the
                      number of updates so far including this one.
* ``lion_step``    -- one Lion iteration, the scalar optimizer of the paper's
                      160M comparison (Sec. 4, "Lion as the scalar optimizer in
                      line with the codebase"); the paper does not print it, so
                      it follows its definition by Chen et al. (2023), with
                      decoupled weight decay and the same clipping:
                          c = b1 m + (1 - b1) g,
                          p <- p (1 - lr wd) - lr sign(c),
                          m <- b2 m + (1 - b2) g.
* ``lr_cosine``, ``lr_wsd`` -- the two schedules.

Readings taken where the paper is silent (listed in the design notes):
the betas (0.9, 0.95) and eps 1e-8 are defaults, not the paper's; the 1e-6 in
the clipping denominator; a linear warmup lr_max (t + 1) / W over the first W
steps of either schedule; cosine from lr_max at the end of warmup to lr_min at
t = T; WSD constant at lr_max until T - D and linear to lr_min at t = T
(D = the cooldown steps; D = 0 never decays); lr_min after T for both.
"""

from __future__ import annotations

import math
from typing import List, Sequence

import numpy as np

CLIP_EPS = 1e-6


def global_norm(grads: Sequence[np.ndarray]) -> float:
    """||g||_2 over every element of every tensor."""
    return math.sqrt(sum(float(np.sum(np.asarray(g, dtype=np.float64) ** 2)) for g in grads))


def clip_factor(grads: Sequence[np.ndarray], max_norm: float) -> float:
    """Scale applied to every gradient by global-norm clipping (1 when off)."""
    if max_norm <= 0:
        return 1.0
    return min(1.0, max_norm / (global_norm(grads) + CLIP_EPS))


def adamw_step(params: List[np.ndarray], grads: Sequence[np.ndarray], m: List[np.ndarray],
               v: List[np.ndarray], t: int, lr: float, beta1: float = 0.9, beta2: float = 0.95,
               eps: float = 1e-8, weight_decay: float = 0.1, max_norm: float = 1.0):
    """One AdamW update of every tensor, t >= 1 counting this update.
    Returns (params, m, v) as new float64 arrays."""
    if t < 1:
        raise ValueError("t counts updates and starts at 1")
    c = clip_factor(grads, max_norm)
    bc1 = 1.0 - beta1 ** t
    bc2 = 1.0 - beta2 ** t
    out_p, out_m, out_v = [], [], []
    for p, g, mi, vi in zip(params, grads, m, v):
        p = np.asarray(p, dtype=np.float64)
        g = c * np.asarray(g, dtype=np.float64)
        mi = beta1 * np.asarray(mi, dtype=np.float64) + (1.0 - beta1) * g
        vi = beta2 * np.asarray(vi, dtype=np.float64) + (1.0 - beta2) * g * g
        p = p * (1.0 - lr * weight_decay)
        p = p - lr * (mi / bc1) / (np.sqrt(vi / bc2) + eps)
        out_p.append(p)
        out_m.append(mi)
        out_v.append(vi)
    return out_p, out_m, out_v


def lion_step(params: List[np.ndarray], grads: Sequence[np.ndarray], m: List[np.ndarray], lr: float,
              beta1: float = 0.9, beta2: float = 0.99, weight_decay: float = 0.1,
              max_norm: float = 1.0):
    """One Lion update of every tensor.  Returns (params, m) as new float64
    arrays.  sign(0) = 0 (numpy's sign; a NaN stays NaN)."""
    c_clip = clip_factor(grads, max_norm)
    out_p, out_m = [], []
    for p, g, mi in zip(params, grads, m):
        p = np.asarray(p, dtype=np.float64)
        g = c_clip * np.asarray(g, dtype=np.float64)
        mi = np.asarray(mi, dtype=np.float64)
        direction = np.sign(beta1 * mi + (1.0 - beta1) * g)
        out_p.append(p * (1.0 - lr * weight_decay) - lr * direction)
        out_m.append(beta2 * mi + (1.0 - beta2) * g)
    return out_p, out_m


def lr_cosine(t: int, total: int, lr_max: float, lr_min: float = 0.0, warmup: int = 0) -> float:
    """Cosine decay from lr_max (end of warmup) to lr_min at t = total."""
    if t < warmup:
        return lr_max * (t + 1) / warmup
    span = max(1, total - warmup)
    x = min(1.0, (t - warmup) / span)
    return lr_min + (lr_max - lr_min) * 0.5 * (1.0 + math.cos(math.pi * x))


def lr_wsd(t: int, total: int, lr_max: float, lr_min: float = 0.0, warmup: int = 0,
           decay: int = 0) -> float:
    """Warmup-stable-decay: linear warmup, constant lr_max, then a linear
    decay over the last ``decay`` steps to lr_min at t = total."""
    if t < warmup:
        return lr_max * (t + 1) / warmup
    if decay <= 0 or t < total - decay:
        return lr_max
    if t >= total:
        return lr_min
    return lr_max + (lr_min - lr_max) * ((t - (total - decay)) / decay)
