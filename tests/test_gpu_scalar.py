"""GPU parity of the scalar optimizer (AdamW with global-norm clipping)
against the fp64 oracle on seeded inputs.

Each step is teacher-forced: the oracle takes one AdamW step from the GPU's
own params and moments (widened to fp64) with the same gradients, so the
comparison isolates one step's arithmetic.  Bars: relative Frobenius error
<= 1e-4 (the fp32 bar) on the moments in every case and on the params with
fp32 params; with bf16 params, the new params against the oracle's rounded
to bf16, within one bf16 rounding of the step's change.
"""

import numpy as np
import pytest

from oracle import scalar_oracle as S
from tests.gpu_harness import announce, rel

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
B1, B2, EPS, WD = 0.9, 0.95, 1e-8, 0.1

# Ragged sizes: single elements, sub-chunk and sub-segment tails, several
# 16384-element segments with a tail.
SIZES = [1, 7, 8, 9, 4096, 16384 + 3, 50000, 3]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2510_16981_amd import muonbp as mb
    mb.load_library()


def _inputs(sizes, seed, dtype, steps, grad_scale):
    import torch
    rng = np.random.default_rng(seed)
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]
    params = [torch.from_numpy(0.02 * rng.standard_normal(n)).to(tdt) for n in sizes]
    grads = [[torch.from_numpy(grad_scale * rng.standard_normal(n) / np.sqrt(n)).to(tdt) for n in sizes]
             for _ in range(steps)]
    return params, grads


def _run(sizes, dtype, max_norm, grad_scale, steps=4, hint=0, offset=0):
    import torch
    from paper_2510_16981_amd import muonbp as mb
    code = {"f32": mb.F32, "bf16": mb.BF16}[dtype]
    opt = mb.AdamW(sizes, mb.adamw_options_default(param_dtype=code, max_grad_norm=max_norm,
                                                   stream_hint=hint))
    params_h, grads_h = _inputs(sizes, 1, dtype, steps, grad_scale)
    # offset > 0: tensors start `offset` elements into a buffer (pointers not
    # 16-byte aligned: the element-wise path).
    bufs = [torch.zeros(n + offset, dtype=p.dtype, device="cuda") for n, p in zip(sizes, params_h)]
    params = [b[offset:] for b in bufs]
    for p, h in zip(params, params_h):
        p.copy_(h)
    worst = {"p": 0.0, "m": 0.0, "v": 0.0, "norm": 0.0}
    lrs = [mb.lr_wsd(t, steps, 1e-2, 1e-3, 0, 2) for t in range(steps)]
    for t in range(steps):
        x0 = [p.double().cpu().numpy() for p in params]
        st = [opt.get_state(i) for i in range(len(sizes))]
        m0 = [m.double().cpu().numpy() for m, _ in st]
        v0 = [v.double().cpu().numpy() for _, v in st]
        g = [gg.cuda() for gg in grads_h[t]]
        g64 = [gg.double().numpy() for gg in grads_h[t]]
        opt.step(params, g, t, lrs[t])
        torch.cuda.synchronize()
        xr, mr, vr = S.adamw_step(x0, g64, m0, v0, t + 1, lrs[t], B1, B2, EPS, WD, max_norm)
        x = [p.double().cpu().numpy() for p in params]
        st = [opt.get_state(i) for i in range(len(sizes))]
        torch.cuda.synchronize()
        m = np.concatenate([a.double().cpu().numpy() for a, _ in st])
        v = np.concatenate([b.double().cpu().numpy() for _, b in st])
        worst["m"] = max(worst["m"], rel(m, np.concatenate(mr)))
        worst["v"] = max(worst["v"], rel(v, np.concatenate(vr)))
        xc, xrc, x0c = np.concatenate(x), np.concatenate(xr), np.concatenate(x0)
        if dtype == "f32":
            worst["p"] = max(worst["p"], rel(xc, xrc))
        else:
            # One bf16 rounding of each new param, measured on the change.
            import torch as _t
            rounded = _t.from_numpy(xrc).to(_t.bfloat16).double().numpy()
            bound = np.linalg.norm(rounded - xrc) * 2 + 1e-3 * np.linalg.norm(xrc - x0c)
            worst["p"] = max(worst["p"], float(np.linalg.norm(xc - xrc) / bound))
        if max_norm > 0:
            n_gpu = opt.grad_norm()
            worst["norm"] = max(worst["norm"], abs(n_gpu - S.global_norm(g64)) / S.global_norm(g64))
    opt.close()
    return worst


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("max_norm,grad_scale", [(0.0, 1.0), (1.0, 0.3), (1.0, 25.0)],
                         ids=["no-clip", "below-clip", "clipped"])
def test_adamw_parity(dtype, max_norm, grad_scale):
    announce(f"adamw {dtype} clip {max_norm} scale {grad_scale}")
    w = _run(SIZES, dtype, max_norm, grad_scale)
    announce(f"worst {w}")
    assert w["m"] <= F32_TOL and w["v"] <= F32_TOL and w["norm"] <= F32_TOL
    assert w["p"] <= (F32_TOL if dtype == "f32" else 1.0)


@pytest.mark.parametrize("hint", [1, 2], ids=["plain", "nontemporal"])
def test_adamw_stream_hints_and_unaligned_pointers(hint):
    announce(f"adamw stream hint {hint}, offset pointers")
    w = _run(SIZES, "bf16", 1.0, 25.0, steps=2, hint=hint)
    assert w["m"] <= F32_TOL and w["v"] <= F32_TOL and w["p"] <= 1.0
    w = _run(SIZES, "f32", 1.0, 25.0, steps=2, hint=hint, offset=1)
    assert w["m"] <= F32_TOL and w["v"] <= F32_TOL and w["p"] <= F32_TOL


def test_adamw_deterministic_and_resumable():
    """Same inputs give bit-identical results; a context resumed from the
    first one's moments continues identically."""
    import torch
    from paper_2510_16981_amd import muonbp as mb
    sizes = [5, 20000, 33]
    params_h, grads_h = _inputs(sizes, 2, "bf16", 3, 25.0)
    runs = []
    for _ in range(2):
        opt = mb.AdamW(sizes)
        p = [h.cuda() for h in params_h]
        for t in range(3):
            opt.step(p, [g.cuda() for g in grads_h[t]], t, 1e-2)
        torch.cuda.synchronize()
        runs.append((opt, p))
    for a, b in zip(runs[0][1], runs[1][1]):
        assert torch.equal(a, b)
    # Resume: a fresh context with the first one's moments, one more step each.
    opt0, p0 = runs[0]
    opt2 = mb.AdamW(sizes)
    for i in range(len(sizes)):
        m, v = opt0.get_state(i)
        opt2.set_state(i, m, v)
    p2 = [x.clone() for x in p0]
    g = [x.cuda() for x in grads_h[0]]
    opt0.step(p0, g, 3, 1e-2)
    opt2.step(p2, g, 3, 1e-2)
    torch.cuda.synchronize()
    for a, b in zip(p0, p2):
        assert torch.equal(a, b)
    for o, _ in runs:
        o.close()
    opt2.close()


# ---------------------------------------------------------------- Lion

L_B1, L_B2 = 0.9, 0.99


def _run_lion(sizes, dtype, max_norm, grad_scale, steps=4, offset=0):
    """Teacher-forced Lion steps against the oracle.  sign(c) is an integer
    decision taken from a float: where the oracle's fp64 c lies within fp32
    rounding of zero either sign is a valid result, so those elements are
    checked only for being p (1 - lr wd) - lr s with s in {-1, 0, 1}; every
    other element is compared with the oracle directly."""
    import torch
    from paper_2510_16981_amd import muonbp as mb
    code = {"f32": mb.F32, "bf16": mb.BF16}[dtype]
    opt = mb.AdamW(sizes, mb.adamw_options_default(param_dtype=code, max_grad_norm=max_norm,
                                                   algorithm=1, beta1=L_B1, beta2=L_B2))
    params_h, grads_h = _inputs(sizes, 4, dtype, steps, grad_scale)
    bufs = [torch.zeros(n + offset, dtype=p.dtype, device="cuda") for n, p in zip(sizes, params_h)]
    params = [b[offset:] for b in bufs]
    for p, h in zip(params, params_h):
        p.copy_(h)
    worst = {"p": 0.0, "m": 0.0, "v": 0.0, "undecided": 0}
    lrs = [mb.lr_wsd(t, steps, 1e-2, 1e-3, 0, 2) for t in range(steps)]
    for t in range(steps):
        x0 = [p.double().cpu().numpy() for p in params]
        m0 = [opt.get_state(i)[0].double().cpu().numpy() for i in range(len(sizes))]
        g64 = [gg.double().numpy() for gg in grads_h[t]]
        opt.step(params, [gg.cuda() for gg in grads_h[t]], t, lrs[t])
        torch.cuda.synchronize()
        xr, mr = S.lion_step(x0, g64, m0, lrs[t], L_B1, L_B2, WD, max_norm)
        st = [opt.get_state(i) for i in range(len(sizes))]
        x = np.concatenate([p.double().cpu().numpy() for p in params])
        m = np.concatenate([a.double().cpu().numpy() for a, _ in st])
        v = np.concatenate([b.double().cpu().numpy() for _, b in st])
        worst["m"] = max(worst["m"], rel(m, np.concatenate(mr)))
        worst["v"] = max(worst["v"], float(np.abs(v).max()))  # Lion never writes v
        # Which elements have a sign fixed beyond fp32 rounding.
        clip = S.clip_factor(g64, max_norm)
        mc, gc = np.concatenate(m0), clip * np.concatenate(g64)
        c = L_B1 * mc + (1 - L_B1) * gc
        slack = 1e-6 * (np.abs(L_B1 * mc) + np.abs((1 - L_B1) * gc)) + 1e-30
        decided = np.abs(c) > slack
        xrc, x0c = np.concatenate(xr), np.concatenate(x0)
        decayed = x0c * (1 - lrs[t] * WD)
        if dtype == "f32":
            err = np.abs(x - xrc)[decided]
            bound = 4e-7 * (np.abs(xrc) + lrs[t])[decided]
        else:
            rounded = torch.from_numpy(xrc).to(torch.bfloat16).double().numpy()
            err = np.abs(x - xrc)[decided]
            bound = (2 * np.abs(rounded - xrc) + 1e-3 * lrs[t])[decided]
        worst["p"] = max(worst["p"], float(np.max(err / bound)) if err.size else 0.0)
        und = ~decided
        worst["undecided"] += int(und.sum())
        if und.any():
            tol = 1e-2 * lrs[t] + (0 if dtype == "f32" else 8e-3 * np.abs(decayed[und]))
            gap = np.min(np.abs(x[und][:, None] - (decayed[und][:, None] - lrs[t] * np.array([-1, 0, 1]))),
                         axis=1)
            assert np.all(gap <= tol), "an undecided element is not p (1 - lr wd) - lr s"
    opt.close()
    return worst


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("max_norm,grad_scale", [(0.0, 1.0), (1.0, 25.0)], ids=["no-clip", "clipped"])
def test_lion_parity(dtype, max_norm, grad_scale):
    announce(f"lion {dtype} clip {max_norm} scale {grad_scale}")
    w = _run_lion(SIZES, dtype, max_norm, grad_scale)
    announce(f"worst {w}")
    assert w["m"] <= F32_TOL and w["v"] == 0.0
    assert w["p"] <= 1.0


def test_lion_unaligned_pointers():
    announce("lion f32 offset pointers")
    w = _run_lion(SIZES, "f32", 1.0, 25.0, steps=2, offset=1)
    assert w["m"] <= F32_TOL and w["p"] <= 1.0


def test_lion_state_has_no_second_moment():
    """A Lion context keeps only m: get_state returns zeros for v, set_state
    ignores it, and a context resumed from m alone continues identically."""
    import torch
    from paper_2510_16981_amd import muonbp as mb
    sizes = [5, 20000, 33]
    params_h, grads_h = _inputs(sizes, 6, "bf16", 2, 25.0)
    o = mb.adamw_options_default(algorithm=1, beta1=L_B1, beta2=L_B2)
    a = mb.AdamW(sizes, o)
    pa = [h.cuda() for h in params_h]
    a.step(pa, [g.cuda() for g in grads_h[0]], 0, 1e-2)
    b = mb.AdamW(sizes, o)
    for i in range(len(sizes)):
        m, v = a.get_state(i)
        torch.cuda.synchronize()
        assert torch.count_nonzero(v) == 0 and torch.count_nonzero(m) > 0
        b.set_state(i, m, torch.full_like(v, 7.0))
    pb = [x.clone() for x in pa]
    g = [x.cuda() for x in grads_h[1]]
    a.step(pa, g, 1, 1e-2)
    b.step(pb, g, 1, 1e-2)
    torch.cuda.synchronize()
    for x, y in zip(pa, pb):
        assert torch.equal(x, y)
    a.close()
    b.close()
