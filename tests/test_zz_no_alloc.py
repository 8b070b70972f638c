"""The allocation-free step (muonbp_step_static) against the context API.

muonbp_step_static runs the same kernels and plans as muonbp_create +
muonbp_step, with its scratch in the library's static device array and the
momentum in the caller's buffer.  Two calls in a row, the second on a
smaller workload (so it finds the first one's tables, partial sums and
split-K counters in the shared scratch array), are compared with contexts
run on the same inputs: params and momentum must agree bit for bit, and the
weights' change also agrees with the fp64 oracle to the bf16 bar (fp32
params and momentum, bf16 NS operands, so that the change is not swamped
by the rounding of the weights).
"""

import numpy as np
import pytest

from oracle import muonbp_oracle as O
from paper_2510_16981_amd import workload as W
from tests.gpu_harness import announce, rel

pytestmark = pytest.mark.gpu

LR_BLOCK, LR_FULL, MU, WD, PERIOD = 0.013, 0.02, 0.95, 0.1, 2
BF16_TOL = 2e-2

# First call: two matrices, ragged tiles, a transposed unit, forced K split
# (counters and partial sums in the scratch array); second call: one
# smaller matrix.
CALLS = [
    ([(520, 1000, 1, 2), (1000, 264, 2, 1)], 0),   # full step (t = 0)
    ([(264, 520, 2, 2)], 1),                       # block step (t = 1)
]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2510_16981_amd import muonbp as mb
    mb.load_library()


def _inputs(mats, t, seed):
    params = [W.quantize(W.init_param(r, c, seed, k), "f32") for k, (r, c, _, _) in enumerate(mats)]
    grads = [W.quantize(W.lowrank_grad(r, c, 16, seed, k, t), "f32")
             for k, (r, c, _, _) in enumerate(mats)]
    return params, grads


@pytest.mark.parametrize("k_split", [0, 2], ids=["planner", "k-split-2"])
def test_static_step_matches_context_step(k_split):
    import torch
    from paper_2510_16981_amd import muonbp as mb
    opts = mb.options_default(k_split=k_split, tile_policy=8 if k_split else 0,
                              param_dtype=mb.F32, state_dtype=mb.F32, ns_dtype=mb.BF16)
    for call, (mats, t) in enumerate(CALLS):
        announce(f"static step call {call}: {mats} t={t} k_split={k_split}")
        info = mb.describe_plan(mats, t % PERIOD == 0, opts)
        assert 0 < info.static_scratch_bytes <= mb.STATIC_SCRATCH_BYTES
        params_h, grads_h = _inputs(mats, t, seed=call)
        # Context path: steps 0..t with the same gradients at step t and
        # zero gradients before it, so both start from the same momentum.
        ctx = mb.MuonBP(mats, PERIOD, LR_BLOCK, LR_FULL, MU, WD, options=opts)
        pc = [p.cuda() for p in params_h]
        gz = [torch.zeros_like(p) for p in pc]
        for s in range(t):
            ctx.step([p.clone() for p in pc], gz, s)
        ctx.step(pc, [g.cuda() for g in grads_h], t)
        torch.cuda.synchronize()
        # Allocation-free path, zero momentum (the zero-gradient steps above
        # leave the context's momentum at zero as well).
        ps = [p.cuda() for p in params_h]
        mom = torch.zeros(sum(r * c for r, c, _, _ in mats), dtype=torch.float32, device="cuda")
        mb.step_static(mats, ps, [g.cuda() for g in grads_h], mom, t, PERIOD, LR_BLOCK, LR_FULL,
                       MU, WD, options=opts)
        torch.cuda.synchronize()
        off = 0
        for k, (r, c, _, _) in enumerate(mats):
            assert torch.equal(ps[k], pc[k]), (call, k)
            m_ctx = ctx.get_momentum(k)
            torch.cuda.synchronize()
            assert torch.equal(mom[off:off + r * c].view(r, c), m_ctx), (call, k)
            off += r * c
        # And the oracle (one step from zero momentum; the decay of the
        # zero-gradient steps is applied to the context's params only, so
        # compare the change of the static path's params).
        orc = O.MuonBPOracle([O.MatrixSpec(*m) for m in mats],
                             O.OracleConfig(period=PERIOD, lr_block=LR_BLOCK, lr_full=LR_FULL,
                                            momentum=MU, weight_decay=WD))
        x0 = [p.double().numpy() for p in params_h]
        ref = orc.step(x0, [g.double().numpy() for g in grads_h], t)
        for k in range(len(mats)):
            d_gpu = ps[k].double().cpu().numpy() - x0[k]
            err = rel(d_gpu, ref[k] - x0[k])
            announce(f"call {call} matrix {k}: update vs oracle {err:.3e}")
            assert err <= BF16_TOL
        ctx.close()


def test_static_step_rejects_a_step_beyond_the_scratch():
    import torch
    from paper_2510_16981_amd import muonbp as mb
    mats = [(4096, 8192, 1, 1)]
    info = mb.describe_plan(mats, True)
    assert info.static_scratch_bytes > mb.STATIC_SCRATCH_BYTES
    p = torch.zeros(4096, 8192, dtype=torch.bfloat16, device="cuda")
    mom = torch.zeros(4096 * 8192, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(mb.MuonBPError) as err:
        mb.step_static(mats, [p], [p], mom, 0, 1, 0.01, 0.02, 0.9, 0.0)
    assert mb.STATUS[err.value.status] == "MUONBP_E_TOO_LARGE"
    assert torch.count_nonzero(p) == 0 and torch.count_nonzero(mom) == 0
