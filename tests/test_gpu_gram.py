"""GPU parity of the Gram-space NS iteration against the fp64 oracle.

Every polynomial of Alg. 2 (App. B) is a polynomial in the Gram matrix of
the iterate it starts from, so the library may run up to three iterations
at a time on S x S matrices only (P_j, then Q_j = P_j Q_{j-1} and A_{j+1} =
(A_j P_j) P_j) and end each such segment with one apply Z <- Q Z: the same
U up to rounding.  The planner does so for bf16 units with S >= 128 and
L >= 1.25 S (option gram_iteration = 0); mode 2 forces it on every unit that
allows it, mode 1 turns it off.  The cases cover transposed and
untransposed units, units that iterate as printed in the same launches,
block and full steps, K = 2 .. 7 (segments of 3, 2 and 1 iterations; the
final Q of a segment in either buffer; three segments, so that the third
reads Z[0] again), per-iteration coefficients and fp32 weights, all at the
bf16 bars of the other parity tests: U teacher-forced against Alg. 2 on the
whole matrix, every unit and every 64 x 64 tile; M and X element by element.
"""

import pytest

from tests.gpu_harness import Case, announce, run_case

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2510_16981_amd import muonbp as mb
    mb.load_library()


def _check(case, want_gram_units):
    from paper_2510_16981_amd import muonbp as mb
    opts = mb.options_default(ns_steps=case.ns_steps, gram_iteration=case.gram_iteration)
    units = [mb.describe_plan(case.mats, full, opts).gram_units for full in (False, True)]
    announce(f"gram-space units (block, full) {units}: {case}")
    assert units == want_gram_units
    w = run_case(case).worst()
    announce(f"worst errors {w}")
    assert w["u"] <= TOL and w["u_unit"] <= TOL and w["u_tile"] <= TOL, w
    assert w["m"] <= TOL and w["x"] <= TOL, w
    assert w["m_ulp"] <= 1.0 and w["x_ulp"] <= 1.0, w


# 1024 x 1280 (S = 1024), its transpose, a 768 x 896 unit that iterates as
# printed (L < 1.25 S), and 2048 x 2560 in two column blocks (blocks 2048 x
# 1280 transposed: S = 1280, L = 2048; the whole matrix: S = 2048, L = 1.25 S).
MIXED = [(1024, 1280, 1, 1), (1280, 1024, 1, 1), (768, 896, 1, 1), (2048, 2560, 1, 2)]


def test_mixed_units_block_and_full():
    _check(Case(mats=MIXED, period=2, steps=4, rank=128, seed=11), [4, 3])


# Units at and just above the Gram-space floor (S = 128 .. 256): 128 x 1024
# and 200 x 600 read the momentum in place, 1024 x 136 is transposed (and
# packed), 120 x 800 lies below the floor (as printed), 256 x 2048 in two
# column blocks reads its 256 x 1024 blocks in place with the matrix's row
# pitch.
SMALL = [(128, 1024, 1, 1), (1024, 136, 1, 1), (200, 600, 1, 1), (120, 800, 1, 1), (256, 2048, 1, 2)]


def test_units_at_the_floor():
    _check(Case(mats=SMALL, period=2, steps=4, rank=32, seed=31), [5, 4])


def test_fp32_weights_and_coefficient_table():
    _check(Case(mats=MIXED[:2], period=1, steps=3, rank=128, seed=12, param="f32", state="f32",
                coeffs=[(3.4445, -4.7750, 2.0315), (3.0, -3.2, 1.2), (2.0, -1.5, 0.5)]), [2, 2])


@pytest.mark.parametrize("k", [2, 3, 4, 7])
def test_iteration_counts(k):
    # Mode 2 on 768-row units (below the automatic threshold).
    _check(Case(mats=[(768, 1536, 1, 1), (1536, 768, 1, 1)], period=1, steps=3, ns_steps=k, rank=128,
                seed=13 + k, gram_iteration=2), [2, 2])


def test_both_modes_agree():
    """The same inputs with the Gram-space iteration on and off: both within
    the bar of the oracle, and of each other."""
    import numpy as np
    from tests.gpu_harness import rel
    base = dict(mats=[(1024, 2048, 1, 1), (2048, 1024, 1, 1)], period=1, steps=2, rank=128, seed=21)
    runs = [run_case(Case(gram_iteration=g, **base), keep_updates=True) for g in (0, 1)]
    for r in runs:
        w = r.worst()
        assert w["u"] <= TOL and w["u_tile"] <= TOL, w
    # U depends on the momentum only, and the momentum on the gradients only:
    # the two runs orthogonalize the same inputs at every step.
    assert sorted(runs[0].updates) == sorted(runs[1].updates) == [0, 1]
    for t in (0, 1):
        for k, (ua, ub) in enumerate(zip(runs[0].updates[t], runs[1].updates[t])):
            d = rel(np.asarray(ua, np.float64), np.asarray(ub, np.float64))
            announce(f"step {t} matrix {k}: U with and without the Gram-space iteration {d:.3e} apart")
            assert d <= TOL
