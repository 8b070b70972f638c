"""The momentum read in place as the NS input, against the packed input.

An untransposed unit whose NS input is the bf16 momentum itself skips the
pack: its first Gram and apply read the momentum window in place and apply
the Frobenius scale of Alg. 2 (App. B) to their sums (s^2 and s).  The
allocation-free entry point takes the pack for every unit when the
caller's momentum does not start on a 16-byte boundary, so the same step
with the momentum one element off such a boundary runs the packed input.
Both must agree with each other and with the fp64 oracle to the bf16 bar,
and leave the same momentum.
"""

import pytest

from oracle import muonbp_oracle as O
from paper_2510_16981_amd import workload as W
from tests.gpu_harness import announce, rel

pytestmark = pytest.mark.gpu

LR_BLOCK, LR_FULL, MU, WD, PERIOD = 0.013, 0.02, 0.95, 0.1, 2
BF16_TOL = 2e-2
# Untransposed units read in place (the Gram-space iteration on 512 x 1024
# and on the ragged 384 x 1024, as printed on the square 512 x 512 blocks),
# beside a transposed unit that is always packed.
MATS = [(512, 1024, 1, 2), (1024, 512, 2, 1), (384, 1024, 1, 1)]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2510_16981_amd import muonbp as mb
    mb.load_library()


@pytest.mark.parametrize("t", [0, 1], ids=["full-step", "block-step"])
def test_in_place_input_matches_packed_input(t):
    import torch
    from paper_2510_16981_amd import muonbp as mb
    opts = mb.options_default(param_dtype=mb.F32, state_dtype=mb.BF16, ns_dtype=mb.BF16)
    full = t % PERIOD == 0
    info = mb.describe_plan(MATS, full, opts)
    total = sum(r * c for r, c, _, _ in MATS)
    assert info.pack_elements < total  # some units are read in place
    params_h = [W.quantize(W.init_param(r, c, 7, k), "f32") for k, (r, c, _, _) in enumerate(MATS)]
    grads_h = [W.quantize(W.lowrank_grad(r, c, 16, 7, k, t), "f32") for k, (r, c, _, _) in enumerate(MATS)]
    out = {}
    for name, offset in (("in place", 0), ("packed", 1)):
        announce(f"in-place input: {name}, t={t}, {MATS}")
        buf = torch.zeros(total + 8, dtype=torch.bfloat16, device="cuda")
        mom = buf[offset:offset + total]
        assert (mom.data_ptr() % 16 == 0) == (offset == 0)
        ps = [p.cuda() for p in params_h]
        mb.step_static(MATS, ps, [g.cuda() for g in grads_h], mom, t, PERIOD, LR_BLOCK, LR_FULL, MU, WD,
                       options=opts)
        torch.cuda.synchronize()
        out[name] = ([p.double().cpu().numpy() for p in ps], mom.clone())
    assert torch.equal(out["in place"][1], out["packed"][1])
    orc = O.MuonBPOracle([O.MatrixSpec(*m) for m in MATS],
                         O.OracleConfig(period=PERIOD, lr_block=LR_BLOCK, lr_full=LR_FULL, momentum=MU,
                                        weight_decay=WD))
    x0 = [p.double().numpy() for p in params_h]
    ref = orc.step(x0, [g.double().numpy() for g in grads_h], t)
    for k in range(len(MATS)):
        d_in = out["in place"][0][k] - x0[k]
        d_pk = out["packed"][0][k] - x0[k]
        e_pair, e_in, e_pk = rel(d_in, d_pk), rel(d_in, ref[k] - x0[k]), rel(d_pk, ref[k] - x0[k])
        announce(f"t={t} matrix {k}: in place vs packed {e_pair:.3e}, vs oracle {e_in:.3e} / {e_pk:.3e}")
        assert e_pair <= BF16_TOL and e_in <= BF16_TOL and e_pk <= BF16_TOL
