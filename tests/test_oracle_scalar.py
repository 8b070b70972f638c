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


# ---------------------------------------------------------------- Lion

def test_lion_reduces_to_sign_descent_without_momentum():
    """beta1 = beta2 = 0: c = g, so the step is p (1 - lr wd) - lr sign(g)
    (clipping scales g and does not change its sign)."""
    rng = np.random.default_rng(3)
    p = [rng.standard_normal(37)]
    g = [rng.standard_normal(37)]
    g[0][5] = 0.0
    out_p, out_m = S.lion_step(p, g, [np.zeros(37)], lr=0.03, beta1=0.0, beta2=0.0,
                               weight_decay=0.1, max_norm=1.0)
    want = p[0] * (1 - 0.03 * 0.1) - 0.03 * np.sign(g[0])
    assert np.allclose(out_p[0], want, rtol=0, atol=1e-15)
    assert out_p[0][5] == p[0][5] * (1 - 0.003)  # sign(0) = 0
    assert np.allclose(out_m[0], S.clip_factor(g, 1.0) * g[0], rtol=0, atol=1e-15)


def test_lion_constant_gradient_closed_form():
    """With a constant gradient g from m = 0, m_t = (1 - b2^t) g, every c has
    the sign of g, and p_T = d^T p_0 - lr sign(g) (1 - d^T) / (1 - d) with
    d = 1 - lr wd."""
    rng = np.random.default_rng(5)
    p0 = rng.standard_normal(20)
    g = rng.standard_normal(20)
    lr, wd, b1, b2, T = 0.01, 0.1, 0.9, 0.99, 12
    p, m = [p0], [np.zeros(20)]
    for _ in range(T):
        p, m = S.lion_step(p, [g], m, lr, b1, b2, wd, max_norm=0.0)
    d = 1 - lr * wd
    assert np.allclose(p[0], d ** T * p0 - lr * np.sign(g) * (1 - d ** T) / (1 - d), rtol=0, atol=1e-13)
    assert np.allclose(m[0], (1 - b2 ** T) * g, rtol=0, atol=1e-14)


def test_lion_zero_gradient_only_decays():
    p0 = np.linspace(-1, 1, 11)
    p, m = [p0], [np.zeros(11)]
    for _ in range(7):
        p, m = S.lion_step(p, [np.zeros(11)], m, lr=0.1, weight_decay=0.2)
    assert np.array_equal(m[0], np.zeros(11))
    assert np.allclose(p[0], (1 - 0.02) ** 7 * p0, rtol=0, atol=1e-15)


def test_lion_momentum_sum_closed_form():
    """m_T = sum_k (1 - b2) b2^(T-k) g_k over the (unclipped) gradients."""
    rng = np.random.default_rng(9)
    gs = [rng.standard_normal(8) for _ in range(6)]
    b2 = 0.99
    m = [np.zeros(8)]
    p = [np.zeros(8)]
    for g in gs:
        p, m = S.lion_step(p, [g], m, lr=0.01, beta2=b2, max_norm=0.0)
    T = len(gs)
    want = sum((1 - b2) * b2 ** (T - 1 - k) * gs[k] for k in range(T))
    assert np.allclose(m[0], want, rtol=0, atol=1e-15)


def test_lion_hand_worked_steps():
    """Three steps worked by hand (b1 = 0.9, b2 = 0.99, lr = 0.1, no decay,
    no clipping): g = 1 gives c = 0.1 > 0; g = -0.5 gives c = 0.009 - 0.05 =
    -0.041 < 0; g = -0.01 gives c = 0.9 * 0.0049 - 0.001 = 0.00341 > 0 (the
    momentum outvotes a small opposite gradient).  m: 0.01, 0.0049, 0.004751."""
    p, m = [np.array([1.0])], [np.array([0.0])]
    seq_p, seq_m = [], []
    for g in (1.0, -0.5, -0.01):
        p, m = S.lion_step(p, [np.array([g])], m, lr=0.1, beta1=0.9, beta2=0.99, weight_decay=0.0,
                           max_norm=0.0)
        seq_p.append(float(p[0][0]))
        seq_m.append(float(m[0][0]))
    assert np.allclose(seq_p, [0.9, 1.0, 0.9], rtol=0, atol=1e-15)
    assert np.allclose(seq_m, [0.01, 0.0049, 0.004751], rtol=0, atol=1e-15)


def test_lion_nan_propagates():
    p, m = S.lion_step([np.zeros(3)], [np.array([1.0, np.nan, -1.0])], [np.zeros(3)], lr=0.1,
                       max_norm=0.0)
    assert np.isnan(p[0][1]) and np.isfinite(p[0][[0, 2]]).all()
