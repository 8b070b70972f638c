"""The Gram-space schedule of the NS iterations equals Alg. 2 (CPU, fp64).

Each iteration of Alg. 2 (App. B) maps X to q(X X^T) X with q(lam) = a + b
lam + c lam^2.  From A_0 = X_0 X_0^T the library's Gram-space schedule runs
up to three iterations at a time on S x S matrices: P_j = q_j(A_j),
Q_j = P_j Q_{j-1}, A_{j+1} = (A_j P_j) P_j, and ends each segment with
X <- Q X; the next segment starts from a fresh Gram of that X.  In exact
arithmetic this is Alg. 2; here both run in fp64 and must agree to rounding
(the GPU tests check the bf16 kernels against the oracle itself).  This
restates the schedule in numpy as a check of its algebra; it is not the
oracle and not the HIP path.
"""

import numpy as np
import pytest

from oracle import muonbp_oracle as O

SEGMENT = 3


def gram_space_ns(G, K, coeffs, eps=O.NS_EPS):
    X = G.T if G.shape[0] > G.shape[1] else G
    X = X / (np.linalg.norm(X) + eps)
    table = O.ns_coefficients(coeffs, K)
    I = np.eye(X.shape[0])
    for k0 in range(0, K, SEGMENT):
        n = min(SEGMENT, K - k0)
        A = X @ X.T
        Q = None
        for j in range(n):
            a, b, c = table[k0 + j]
            P = a * I + b * A + c * (A @ A)
            Q = P if Q is None else P @ Q
            if j + 1 < n:
                A = (A @ P) @ P
        X = Q @ X
    return X.T if G.shape[0] > G.shape[1] else X


@pytest.mark.parametrize("shape", [(7, 30), (30, 7), (64, 64), (40, 100), (100, 40), (1, 9)])
@pytest.mark.parametrize("K", [1, 2, 3, 4, 5, 7])
def test_gram_space_schedule_equals_algorithm_2(shape, K):
    rng = np.random.default_rng([len(shape), shape[0], shape[1], K])
    G = rng.standard_normal(shape)
    for coeffs in [(O.NS_A, O.NS_B, O.NS_C),
                   [(3.4445, -4.7750, 2.0315), (3.0, -3.2, 1.2), (2.0, -1.5, 0.5)]]:
        ref = O.orthogonalize_via_ns(G, K=K, coeffs=coeffs)
        got = gram_space_ns(G, K, coeffs)
        assert np.linalg.norm(got - ref) <= 1e-11 * max(1.0, np.linalg.norm(ref))


def test_segment_products_commute():
    """The products the kernels compute on upper tiles only are symmetric:
    P, A, Q are polynomials in one Gram matrix, so A P and P Q are."""
    rng = np.random.default_rng(3)
    X = rng.standard_normal((20, 50))
    X /= np.linalg.norm(X)
    A = X @ X.T
    P = 2.0 * np.eye(20) - 1.5 * A + 0.5 * A @ A
    Q = P @ (2.0 * np.eye(20) - 1.5 * A)
    for M in (A @ P, P @ Q, (A @ P) @ P):
        assert np.allclose(M, M.T, rtol=0, atol=1e-13)
