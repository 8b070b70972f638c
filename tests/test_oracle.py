"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these retypes the oracle's formulas: the NS output is checked against
a closed form built from a LAPACK SVD, the polar factor, the paper's norm
lemmas, closed forms of momentum and weight decay, and the paper's own worked
FLOP example.  Each test names the passage it relies on.
"""

import json
import math
import os

import numpy as np
import pytest

from oracle import muonbp_oracle as O
from paper_2510_16981_amd import workload as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _phi(x, K, a=O.NS_A, b=O.NS_B, c=O.NS_C):
    """K-fold composition of the scalar quintic p(x) = a x + b x^3 + c x^5."""
    for _ in range(K):
        x = a * x + b * x ** 3 + c * x ** 5
    return x


def _svd_closed_form(Z, K, eps=O.NS_EPS, coeffs=(O.NS_A, O.NS_B, O.NS_C)):
    """Each NS iteration is an odd matrix polynomial, so it keeps the singular
    vectors and maps each singular value sigma/(||Z||_F+eps) through phi_K."""
    U, s, Vt = np.linalg.svd(Z, full_matrices=False)
    x = s / (np.linalg.norm(s) + eps)
    return (U * _phi(x, K, *coeffs)) @ Vt


def _rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


SHAPES = [(8, 5), (5, 8), (16, 16), (3, 1), (1, 4), (1, 1), (32, 7), (7, 33)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("K", [0, 1, 3, 5, 8])
def test_ns_matches_svd_closed_form(shape, K):
    """Alg. 2 vs its spectral closed form (Sec. 2.2 defines Orth via the SVD)."""
    rng = np.random.default_rng(hash((shape, K)) % 2**32)
    Z = rng.standard_normal(shape) * 3.7
    got = O.orthogonalize_via_ns(Z, K=K)
    want = _svd_closed_form(Z, K)
    assert _rel(got, want) <= 1e-12


def test_ns_closed_form_other_coefficients():
    """Alg. 2 with arbitrary (a, b, c): the closed form still holds, so a
    swapped or dropped coefficient cannot pass."""
    rng = np.random.default_rng(1)
    Z = rng.standard_normal((6, 11))
    coeffs = (3.4445, -4.7750, 2.0315)
    got = O.orthogonalize_via_ns(Z, K=4, coeffs=coeffs)
    assert _rel(got, _svd_closed_form(Z, 4, coeffs=coeffs)) <= 1e-12


def test_ns_closed_form_per_iteration_coefficients():
    """Iteration k with its own (a_k, b_k, c_k): each step is still an odd
    matrix polynomial, so the closed form composes p_K o ... o p_1 on the
    singular values.  A table shorter than K repeats its last entry; a table
    of one entry is the constant quintic."""
    rng = np.random.default_rng(7)
    Z = rng.standard_normal((9, 14))
    table = [(4.0, -5.0, 1.5), (3.4445, -4.7750, 2.0315), (2.0, -1.5, 0.5)]
    U, s, Vt = np.linalg.svd(Z, full_matrices=False)
    x = s / (np.linalg.norm(s) + O.NS_EPS)
    for a, b, c in table + [table[-1]] * 2:  # K = 5: the last entry twice more
        x = a * x + b * x ** 3 + c * x ** 5
    want = (U * x) @ Vt
    assert _rel(O.orthogonalize_via_ns(Z, K=5, coeffs=table), want) <= 1e-12
    # Order matters (the p_k do not commute), so a reversed table differs.
    assert _rel(O.orthogonalize_via_ns(Z, K=5, coeffs=table[::-1]), want) > 1e-3
    assert np.array_equal(O.orthogonalize_via_ns(Z, K=3, coeffs=[(2.0, -1.5, 0.5)]),
                          O.orthogonalize_via_ns(Z, K=3))
    with pytest.raises(ValueError):
        O.ns_coefficients([(1.0, 2.0)], 2)


def test_ns_singular_value_band():
    """p(x) = 2x - 1.5x^3 + 0.5x^5 has p(1) = 1, p'(1) = 0 and its maximum on
    [0, 1] at x^2 = 0.8, where p = 1.12 sqrt(0.8).  The Frobenius
    pre-normalisation puts every ratio in [0, 1], so every output singular
    value lies in [0, 1.12 sqrt(0.8)] and small ones grow by 2 per step."""
    pmax = 1.12 * math.sqrt(0.8)
    assert abs(_phi(math.sqrt(0.8), 1) - pmax) < 1e-15
    assert abs(_phi(1.0, 1) - 1.0) < 1e-15
    xs = np.linspace(0, 1, 100001)
    assert _phi(xs, 1).max() <= pmax + 1e-15
    rng = np.random.default_rng(2)
    for shape in [(12, 40), (40, 12), (30, 30)]:
        Z = rng.standard_normal(shape) @ np.diag(np.logspace(0, -3, shape[1]))
        s_out = np.linalg.svd(O.orthogonalize_via_ns(Z, K=5), compute_uv=False)
        assert s_out.max() <= pmax + 1e-12
        assert s_out.min() >= -1e-12
    # Ratios >= 0.0588 reach >= 0.99 after five steps.
    assert _phi(0.0588, 5) >= 0.99
    # Small-sigma gain is a^K = 32.
    assert abs(_phi(1e-9, 5) / 1e-9 - 32.0) < 1e-6


def test_ns_converges_to_polar_factor():
    """Orth(G) = (G G^T)^{-+/2} G = U V^T (Sec. 2.2, eq. (1)); with many
    iterations NS reaches it, for wide and tall inputs."""
    rng = np.random.default_rng(3)
    for shape in [(6, 10), (10, 6), (9, 9)]:
        Q1, _ = np.linalg.qr(rng.standard_normal((shape[0], shape[0])))
        Q2, _ = np.linalg.qr(rng.standard_normal((shape[1], shape[1])))
        r = min(shape)
        s = np.linspace(1.0, 0.5, r)
        Z = (Q1[:, :r] * s) @ Q2[:, :r].T
        U, _, Vt = np.linalg.svd(Z, full_matrices=False)
        assert _rel(O.orthogonalize_via_ns(Z, K=40), U @ Vt) <= 1e-10


def test_ns_rank_deficient_polar_uses_pseudo_inverse():
    """The pseudo-inverse in Orth maps the null space to zero.  K stays at
    20: rounding noise on the null space (~1e-16) grows by 2 per step."""
    rng = np.random.default_rng(4)
    Q1, _ = np.linalg.qr(rng.standard_normal((8, 3)))
    Q2, _ = np.linalg.qr(rng.standard_normal((12, 3)))
    Z = (Q1 * np.array([1.0, 0.8, 0.6])) @ Q2.T  # rank 3
    polar = Q1 @ Q2.T
    got = O.orthogonalize_via_ns(Z, K=20)
    assert _rel(got, polar) <= 1e-8
    assert np.linalg.matrix_rank(got, tol=1e-6) == 3


def test_transpose_rule_is_exact_in_exact_arithmetic():
    """Running NS on G^T and transposing back equals running it on G."""
    rng = np.random.default_rng(5)
    Z = rng.standard_normal((37, 9))
    direct = O.orthogonalize_via_ns(Z, K=5, transpose_tall=False)
    via_t = O.orthogonalize_via_ns(Z, K=5, transpose_tall=True)
    assert _rel(via_t, direct) <= 1e-13


def test_zero_input_gives_zero():
    """Lemma (dual of the block-spectral norm): a zero block maps to 0."""
    assert np.all(O.orthogonalize_via_ns(np.zeros((4, 6)), K=5) == 0.0)


@pytest.mark.parametrize("t,P,want", [(0, 1, True), (7, 1, True), (0, 5, True),
                                      (4, 5, False), (5, 5, True), (10, 5, True),
                                      (0, 0, False), (5, 0, False)])
def test_scheduler_cases(t, P, want):
    assert O.is_full_step(t, P) is want


def test_scheduler_truth_table():
    """Alg. 1: full iff t mod P == 0; P = 1 is Muon (every step full) and
    P -> infinity is BlockMuon (never full), Sec. 3.2."""
    for P in (1, 2, 5, 10):
        fulls = [t for t in range(100) if O.is_full_step(t, P)]
        assert fulls == list(range(0, 100, P))
        assert len(fulls) == 100 // P
    assert not any(O.is_full_step(t, 0) for t in range(100))
    with pytest.raises(ValueError):
        O.is_full_step(-1, 5)


def test_block_ranges_partition():
    """Sec. 3 shard grid: blocks tile the matrix exactly once."""
    m, n, r, c = 12, 20, 3, 4
    cover = np.zeros((m, n), int)
    for rs, cs in O.block_ranges(m, n, r, c):
        assert (rs.stop - rs.start, cs.stop - cs.start) == (4, 5)
        cover[rs, cs] += 1
    assert np.all(cover == 1)
    with pytest.raises(ValueError):
        O.block_ranges(10, 10, 3, 1)


def test_blockwise_is_concatenation_of_blocks():
    """BlockMuon orthogonalizes each shard independently (Sec. 3.1)."""
    rng = np.random.default_rng(6)
    M = rng.standard_normal((12, 20))
    U = O.orthogonalize_blockwise(M, (2, 4), K=5)
    rows = []
    for i in range(2):
        rows.append(np.hstack([
            _svd_closed_form(M[6 * i:6 * i + 6, 5 * j:5 * j + 5], 5)
            for j in range(4)]))
    assert _rel(U, np.vstack(rows)) <= 1e-12


def test_grid_1x1_block_step_equals_full_step():
    rng = np.random.default_rng(7)
    M = rng.standard_normal((9, 14))
    assert np.array_equal(O.orthogonalize_blockwise(M, (1, 1)),
                          O.orthogonalize_via_ns(M))


def test_column_blocks_are_column_normalisation():
    """Sec. 2.2: orthogonalising m x 1 blocks is column normalisation."""
    rng = np.random.default_rng(8)
    M = rng.standard_normal((10, 6))
    U = O.orthogonalize_blockwise(M, (1, 6), K=30)
    norms = np.linalg.norm(M, axis=0)
    assert _rel(U, M / norms) <= 1e-12
    # Finite K: the single singular value x = ||g|| / (||g|| + eps) maps to
    # phi_K(x) along the unit direction g / ||g||.
    U5 = O.orthogonalize_blockwise(M, (1, 6), K=5)
    x = norms / (norms + O.NS_EPS)
    assert _rel(U5, M / norms * _phi(x, 5)) <= 1e-12


def test_block_norm_invariants_at_polar_limit():
    """Lemmas of App. A.1: Z*_ij = U_ij V_ij^T attains <M, Z*> = sum of block
    nuclear norms, has B(Z*) = 1, and ||Z*||_op <= sqrt(rc) B(Z*)."""
    rng = np.random.default_rng(9)
    m, n, r, c = 16, 24, 2, 3
    M = rng.standard_normal((m, n))
    U = O.orthogonalize_blockwise(M, (r, c), K=40)
    nuc = sum(np.linalg.norm(M[rs, cs], "nuc") for rs, cs in O.block_ranges(m, n, r, c))
    assert abs(np.sum(M * U) - nuc) <= 1e-9 * nuc
    assert nuc >= np.linalg.norm(M, "nuc") - 1e-9
    B = max(np.linalg.norm(U[rs, cs], 2) for rs, cs in O.block_ranges(m, n, r, c))
    assert abs(B - 1.0) <= 1e-9
    assert np.linalg.norm(U, 2) <= math.sqrt(r * c) * B + 1e-9


def test_momentum_closed_form():
    """eq. (NTR) / Alg. 1 with M_{-1} = 0: M_t = sum_k mu^{t-k} G_k."""
    rng = np.random.default_rng(10)
    mu = 0.95
    Gs = [rng.standard_normal((4, 5)) for _ in range(7)]
    M = np.zeros((4, 5))
    for t, G in enumerate(Gs):
        M = O.momentum_update(M, G, mu)
        want = sum(mu ** (t - k) * Gs[k] for k in range(t + 1))
        assert _rel(M, want) <= 1e-12


def _cfg(**kw):
    base = dict(period=3, lr_block=0.013, lr_full=0.029, momentum=0.9,
                weight_decay=0.1, ns_steps=5)
    base.update(kw)
    return O.OracleConfig(**base)


def test_zero_gradients_decay_with_the_step_kinds_lr():
    """With G = 0, U = 0 and each step scales X by (1 - eta_t lambda): the two
    stepsizes of Alg. 1 are applied on their own step kinds."""
    spec = [O.MatrixSpec(6, 8, 2, 2)]
    cfg = _cfg()
    orc = O.MuonBPOracle(spec, cfg)
    X0 = np.random.default_rng(11).standard_normal((6, 8))
    X = [X0]
    T = 9
    for t in range(T):
        X = orc.step(X, [np.zeros((6, 8))], t)
    nfull = sum(O.is_full_step(t, cfg.period) for t in range(T))
    f = (1 - cfg.lr_full * cfg.weight_decay) ** nfull * \
        (1 - cfg.lr_block * cfg.weight_decay) ** (T - nfull)
    assert _rel(X[0], f * X0) <= 1e-12


def test_step_composition_against_closed_forms():
    """Alg. 1 end to end for two steps (t = 0 full, t = 1 block) with
    lambda = 0: X_{t+1} - X_t = -eta_t Orth_NS(M_t), each checked against the
    SVD closed form, so the sign, the NS input (M, not G) and the stepsize
    choice are all pinned."""
    rng = np.random.default_rng(12)
    spec = [O.MatrixSpec(8, 12, 1, 3)]
    cfg = _cfg(period=2, weight_decay=0.0)
    orc = O.MuonBPOracle(spec, cfg)
    X0 = rng.standard_normal((8, 12))
    G0, G1 = rng.standard_normal((8, 12)), rng.standard_normal((8, 12))
    X1 = orc.step([X0], [G0], 0)[0]
    assert _rel(X0 - X1, cfg.lr_full * _svd_closed_form(G0, 5)) <= 1e-12
    X2 = orc.step([X1], [G1], 1)[0]
    M1 = cfg.momentum * G0 + G1
    U1 = np.hstack([_svd_closed_form(M1[:, 4 * j:4 * j + 4], 5) for j in range(3)])
    assert _rel(X1 - X2, cfg.lr_block * U1) <= 1e-12


def test_nesterov_input_closed_form():
    """The Nesterov variant (an opt-in reading: the paper's Alg. 1 has the
    heavy-ball sum only): the NS input is G_t + mu M_t, M_t being the
    momentum after this step's update.  With lambda = 0, two steps from
    M = 0 have closed forms, Y_0 = (1 + mu) G_0 and Y_1 = (1 + mu) G_1 +
    mu^2 G_0, each update being the SVD closed form of its input.  Taking
    the momentum before the update (Y_1 = G_1 + mu G_0) or dropping mu fails
    here."""
    rng = np.random.default_rng(13)
    spec = [O.MatrixSpec(8, 12, 1, 3)]
    cfg = _cfg(period=2, weight_decay=0.0, nesterov=True)
    mu = cfg.momentum
    orc = O.MuonBPOracle(spec, cfg)
    X0 = rng.standard_normal((8, 12))
    G0, G1 = rng.standard_normal((8, 12)), rng.standard_normal((8, 12))
    X1 = orc.step([X0], [G0], 0)[0]
    assert _rel(X0 - X1, cfg.lr_full * _svd_closed_form((1 + mu) * G0, 5)) <= 1e-12
    X2 = orc.step([X1], [G1], 1)[0]
    Y1 = (1 + mu) * G1 + mu ** 2 * G0
    U1 = np.hstack([_svd_closed_form(Y1[:, 4 * j:4 * j + 4], 5) for j in range(3)])
    assert _rel(X1 - X2, cfg.lr_block * U1) <= 1e-12


def test_period_one_is_muon_and_infinite_period_is_blockmuon():
    """Sec. 3.2: P = 1 gives Muon (every step full), P = infinity gives
    BlockMuon (every step blockwise)."""
    rng = np.random.default_rng(13)
    spec = [O.MatrixSpec(6, 9, 2, 3)]
    Gs = [rng.standard_normal((6, 9)) for _ in range(4)]
    X0 = rng.standard_normal((6, 9))
    for period, full in [(1, True), (0, False)]:
        orc = O.MuonBPOracle(spec, _cfg(period=period, weight_decay=0.0))
        X = [X0]
        M = np.zeros((6, 9))
        Xref = X0.copy()
        for t, G in enumerate(Gs):
            X = orc.step(X, [G], t)
            M = 0.9 * M + G
            if full:
                U = _svd_closed_form(M, 5)
                eta = 0.029
            else:
                U = np.vstack([np.hstack([
                    _svd_closed_form(M[3 * i:3 * i + 3, 3 * j:3 * j + 3], 5)
                    for j in range(3)]) for i in range(2)])
                eta = 0.013
            Xref = Xref - eta * U
        assert _rel(X[0], Xref) <= 1e-12


def test_rms_matching_gives_update_rms_beta():
    """Sec. 3.2 (AdamW learning rate transfer): scaling an orthogonal update
    of a p x q unit by beta sqrt(max(p, q)) makes its RMS equal beta.  The
    unit is the block on block steps and the matrix on full steps."""
    rng = np.random.default_rng(14)
    spec = [O.MatrixSpec(8, 24, 1, 2)]
    beta = 0.2
    for t, shape in [(0, (8, 24)), (1, (8, 12))]:
        orc = O.MuonBPOracle(spec, _cfg(period=2, scale_mode=1, rms_beta=beta,
                                        ns_steps=40, weight_decay=0.0))
        G = rng.standard_normal((8, 24))
        if t == 1:
            orc.step([np.zeros((8, 24))], [np.zeros((8, 24))], 0)
        _, rec = orc.step([np.zeros((8, 24))], [G], t, record=True)
        U = rec.U[0]
        assert rec.full is (t == 0)
        rms = np.sqrt(np.mean(U ** 2))
        assert abs(rms - beta) <= 1e-9


def test_paper_flop_example():
    """Sec. 3 first bullet: 8-way TP blocks cut the per-NS-step cost of the
    Llama 3 405B MLP matrices by about 2.36x (up) and 9.06x (down)."""
    with open(os.path.join(GOLDEN, "paper_flop_example.json")) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        m, n = case["full"]
        r, c = case["grid"]
        assert [m // r, n // c] == case["block"]
        ratio = O.ns_dense_flops(m, n, 1) / O.ns_blockwise_dense_flops(m, n, r, c, 1)
        assert round(ratio, 2) == case["speedup"]
    # The blockwise form 2(2mnq + mnq^2/p) of the same bullet (p <= q), with
    # q = the larger block side here, reproduces the per-block sum.
    m, n = 16384, 53248
    q, p = 16384, 6656
    assert abs(O.ns_blockwise_dense_flops(m, n, 1, 8, 1)
               - 2 * (2 * m * n * p + m * n * p * p / q)) < 1.0


def test_workload_generator_spectrum():
    """The synthetic gradient has the stated spectrum: s_i = 1/i plus small
    noise, and X_0 has std 0.02."""
    G = W.lowrank_grad(256, 512, 32, seed=0, k=0, t=0)
    s = np.linalg.svd(G, compute_uv=False)
    assert np.allclose(s[:8], 1.0 / np.arange(1, 9), atol=0.05)
    assert s[40] < 0.05
    X = W.init_param(256, 512, seed=0, k=0)
    assert abs(X.std() - 0.02) < 1e-3
    # Each (k, t) stream is independent and reproducible.
    assert np.array_equal(W.lowrank_grad(16, 8, 4, 0, 3, 5),
                          W.lowrank_grad(16, 8, 4, 0, 3, 5))
    assert not np.array_equal(W.lowrank_grad(16, 8, 4, 0, 3, 5),
                              W.lowrank_grad(16, 8, 4, 0, 3, 6))
