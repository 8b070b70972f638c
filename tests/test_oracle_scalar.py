"""Pins of the scalar-optimizer and schedule oracle (CPU only).

AdamW and clipping are pinned to torch's own CPU implementations in float64
(torch.optim.AdamW, torch.nn.utils.clip_grad_norm_: the library routines the
definitions reduce to) and to closed forms of Adam's bias correction; the
schedules to their values at the phase boundaries.
"""

import math

import numpy as np
import pytest

from oracle import scalar_oracle as S

B1, B2, EPS, WD = 0.9, 0.95, 1e-8, 0.1


def _tensors(seed, sizes=(7, 1, 33, 100)):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal(n) for n in sizes]


def test_adamw_matches_torch_adamw_fp64():
    import torch
    p0 = _tensors(0)
    grads = [_tensors(10 + t) for t in range(6)]
    lrs = [1e-2, 2e-2, 5e-3, 1e-3, 3e-2, 1e-2]
    tp = [torch.tensor(p, dtype=torch.float64, requires_grad=True) for p in p0]
    opt = torch.optim.AdamW(tp, lr=1.0, betas=(B1, B2), eps=EPS, weight_decay=WD)
    p = [x.copy() for x in p0]
    m = [np.zeros_like(x) for x in p0]
    v = [np.zeros_like(x) for x in p0]
    for t in range(6):
        for x, g in zip(tp, grads[t]):
            x.grad = torch.tensor(g, dtype=torch.float64)
        for group in opt.param_groups:
            group["lr"] = lrs[t]
        opt.step()
        p, m, v = S.adamw_step(p, grads[t], m, v, t + 1, lrs[t], B1, B2, EPS, WD, max_norm=0.0)
        for x, y in zip(tp, p):
            np.testing.assert_allclose(x.detach().numpy(), y, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("scale", [0.01, 1.0, 50.0])
def test_clipping_matches_torch_clip_grad_norm(scale):
    import torch
    grads = [scale * g for g in _tensors(3)]
    tg = [torch.tensor(g, dtype=torch.float64) for g in grads]
    params = [torch.zeros_like(g, requires_grad=True) for g in tg]
    for p, g in zip(params, tg):
        p.grad = g.clone()
    torch.nn.utils.clip_grad_norm_(params, max_norm=1.0)
    c = S.clip_factor(grads, 1.0)
    for p, g in zip(params, grads):
        np.testing.assert_allclose(p.grad.numpy(), c * g, rtol=1e-14, atol=0)
    clipped = S.global_norm([c * g for g in grads])
    if S.global_norm(grads) > 1.0:
        assert abs(clipped - 1.0) < 1e-5
    else:
        assert c == 1.0


def test_first_step_closed_form():
    """t = 1: m_hat = g and v_hat = g^2, so with eps = 0 the step is
    lr (wd p + sign(g))."""
    p0, g = _tensors(4), _tensors(5)
    lr = 0.03
    p, _, _ = S.adamw_step(p0, g, [0 * x for x in p0], [0 * x for x in p0], 1, lr, B1, B2, 0.0, WD,
                           max_norm=0.0)
    for x0, gi, x in zip(p0, g, p):
        np.testing.assert_allclose(x, x0 * (1 - lr * WD) - lr * np.sign(gi), rtol=1e-14, atol=1e-16)


def test_constant_gradient_has_exact_bias_correction():
    """With the same gradient at every step, m_hat = g and v_hat = g^2 at
    every t (the bias correction undoes the zero start exactly)."""
    g = _tensors(6)
    p = _tensors(7)
    m = [0 * x for x in p]
    v = [0 * x for x in p]
    lr = 0.01
    for t in range(1, 30):
        before = [x.copy() for x in p]
        p, m, v = S.adamw_step(p, g, m, v, t, lr, B1, B2, EPS, WD, max_norm=0.0)
        for mi, vi, gi in zip(m, v, g):
            np.testing.assert_allclose(mi / (1 - B1 ** t), gi, rtol=1e-12)
            np.testing.assert_allclose(vi / (1 - B2 ** t), gi * gi, rtol=1e-12)
        for x0, x, gi in zip(before, p, g):
            np.testing.assert_allclose(x, x0 * (1 - lr * WD) - lr * gi / (np.abs(gi) + EPS),
                                       rtol=1e-12, atol=1e-15)


def test_zero_gradient_only_decays():
    p0 = _tensors(8)
    p = [x.copy() for x in p0]
    m = [0 * x for x in p0]
    v = [0 * x for x in p0]
    lr = 0.02
    for t in range(1, 11):
        p, m, v = S.adamw_step(p, [0 * x for x in p0], m, v, t, lr, B1, B2, EPS, WD, max_norm=1.0)
    for x0, x in zip(p0, p):
        np.testing.assert_allclose(x, x0 * (1 - lr * WD) ** 10, rtol=1e-13)


def test_cosine_schedule_boundaries():
    T, hi, lo = 1000, 3e-3, 3e-5
    assert S.lr_cosine(0, T, hi, lo) == hi
    assert abs(S.lr_cosine(T, T, hi, lo) - lo) < 1e-18
    assert S.lr_cosine(T + 50, T, hi, lo) == lo
    assert abs(S.lr_cosine(T // 2, T, hi, lo) - (hi + lo) / 2) < 1e-15
    assert abs(S.lr_cosine(T // 4, T, hi, lo) - (lo + (hi - lo) * (1 + math.cos(math.pi / 4)) / 2)) < 1e-15
    vals = [S.lr_cosine(t, T, hi, lo) for t in range(T + 1)]
    assert all(a >= b for a, b in zip(vals, vals[1:]))
    # Warmup: linear up to lr_max at the last warmup step, then the decay.
    assert S.lr_cosine(0, T, hi, lo, warmup=10) == hi / 10
    assert S.lr_cosine(9, T, hi, lo, warmup=10) == hi
    assert S.lr_cosine(10, T, hi, lo, warmup=10) == hi


def test_wsd_schedule_boundaries():
    """The 160M setting: no warmup, 20% cooldown, linear to the final lr."""
    T, hi, lo = 1000, 2e-2, 4.2e-5
    D = T // 5
    assert all(S.lr_wsd(t, T, hi, lo, 0, D) == hi for t in range(0, T - D + 1))
    assert abs(S.lr_wsd(T - D // 2, T, hi, lo, 0, D) - (hi + lo) / 2) < 1e-15
    assert abs(S.lr_wsd(T, T, hi, lo, 0, D) - lo) < 1e-18
    assert S.lr_wsd(T + 7, T, hi, lo, 0, D) == lo
    assert S.lr_wsd(T, T, hi, lo, 0, 0) == hi
    assert S.lr_wsd(3, T, hi, lo, warmup=4, decay=D) == hi
    assert S.lr_wsd(1, T, hi, lo, warmup=4, decay=D) == hi / 2
