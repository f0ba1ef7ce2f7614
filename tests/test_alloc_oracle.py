"""Pins of the mixed-bit allocation oracle (Sec. 4.3, Eq. 3-4), CPU only.

Criterion: closed forms for calibration sets whose Gram matrix is diagonal
(then diag(cholesky(H^{-1})) = 1/sqrt(diag H)), the scaling law of X (IS scales
with X, C with its cube), the reversed-order Cholesky identity (the diagonal
of the Cholesky factor of H^{-1} is the reversed reciprocal diagonal of the
Cholesky factor of the reversed H, a fact about triangular factors), and
brute-force agreement with explicit conditional variances.  Fit: exact
recovery of polynomials.  Allocation: hand cases, budget extremes, the tie
rule, and a planted mistake.
"""
import numpy as np
import pytest

from oracle import alloc


def test_diagonal_gram_closed_form():
    rng = np.random.default_rng(0)
    K, T = 16, 64
    # orthogonal rows: X X^T = diag(s)
    Q, _ = np.linalg.qr(rng.standard_normal((T, K)))
    s = rng.uniform(0.5, 3.0, K)
    x = (Q * np.sqrt(s)).T                     # [K][T]
    H = alloc.gram(x)
    assert np.allclose(H, np.diag(s), atol=1e-12)
    damp = 0.01
    d = alloc.cholesky_diag_of_inverse(alloc.damped(H, damp))
    assert np.allclose(d, 1.0 / np.sqrt(s + damp * s.mean()), rtol=1e-12)
    w = rng.standard_normal((8, K))
    IS = w * np.sqrt(s + damp * s.mean())[None, :]
    C = np.linalg.norm(IS) * IS.std() ** 2
    assert alloc.criterion(w, x, damp) == pytest.approx(C, rel=1e-12)


def test_scaling_law():
    rng = np.random.default_rng(1)
    w = rng.standard_normal((12, 24))
    x = rng.standard_normal((24, 200))
    c1 = alloc.criterion(w, x)
    c2 = alloc.criterion(w, 3.0 * x)
    assert c2 == pytest.approx(27.0 * c1, rel=1e-9)
    assert np.allclose(alloc.importance(w, 3.0 * x), 3.0 * alloc.importance(w, x), rtol=1e-9)


def test_reversed_cholesky_identity():
    """diag(chol(H^{-1}))[k] = 1 / diag(chol(J H J))[K-1-k], J the reversal."""
    rng = np.random.default_rng(2)
    A = rng.standard_normal((30, 60))
    H = alloc.damped(alloc.gram(A), 0.01)
    lhs = alloc.cholesky_diag_of_inverse(H)
    rhs = 1.0 / np.diag(np.linalg.cholesky(H[::-1, ::-1]))[::-1]
    assert np.allclose(lhs, rhs, rtol=1e-10)


def test_conditional_variance_brute_force():
    """The k-th diagonal entry of chol(H^{-1}) is 1/sqrt(S_k), S_k the Schur
    complement of H on the columns after k (the variance of column k left
    after regressing on the later columns)."""
    rng = np.random.default_rng(3)
    A = rng.standard_normal((8, 40))
    H = alloc.damped(alloc.gram(A), 0.05)
    d = alloc.cholesky_diag_of_inverse(H)
    K = H.shape[0]
    for k in range(K):
        later = list(range(k + 1, K))
        S = H[k, k] - (H[k, later] @ np.linalg.solve(H[np.ix_(later, later)], H[later, k])
                       if later else 0.0)
        assert d[k] == pytest.approx(1.0 / np.sqrt(S), rel=1e-10)


@pytest.mark.parametrize("degree", [1, 2, 3])
def test_fit_recovers_polynomials(degree):
    rng = np.random.default_rng(4)
    c = rng.uniform(0.1, 2.0, 12)
    coefs = rng.standard_normal((3, degree + 1))
    errors = np.stack([np.polyval(coefs[b], c) for b in range(3)], axis=1)
    est = alloc.fit_per_bit(c, errors, degree)
    assert np.allclose(est, errors, rtol=1e-9, atol=1e-12)


def test_allocate_hand_cases():
    bits = [2, 3, 4]
    cost = np.array([[10.0, 4.0, 1.0],    # a sensitive layer
                     [2.0, 1.5, 1.0],     # an insensitive one
                     [6.0, 3.0, 2.0]])
    w, obj = alloc.allocate(cost, bits, budget=3.0)   # 9 bits for 3 layers
    # candidates with 9 bits: (4,2,3)=1+2+3=6, (3,2,4)=4+2+2=8, (4,3,2)=1+1.5+6=8.5,
    # (3,3,3)=4+1.5+3=8.5, (2,3,4)..., best (4,2,3) = 6
    assert w.tolist() == [4, 2, 3] and obj == 6.0
    w, _ = alloc.allocate(cost, bits, budget=4.0)
    assert w.tolist() == [4, 4, 4]
    w, _ = alloc.allocate(cost, bits, budget=2.0)
    assert w.tolist() == [2, 2, 2]
    with pytest.raises(ValueError):
        alloc.allocate(cost, bits, budget=1.5)


def test_allocate_tie_rule():
    bits = [2, 3, 4]
    cost = np.array([[1.0, 1.0, 1.0], [2.0, 1.0, 1.0]])
    # objective 2 by (2,3), (2,4), (3,3), (3,4), (4,3), (4,4) ...: fewest bits (5) -> (2,3)
    w, obj = alloc.allocate(cost, bits, budget=4.0)
    assert w.tolist() == [2, 3] and obj == 2.0
    cost = np.array([[1.0, 0.5, 0.5], [0.5, 1.0, 1.0]])
    # objective 1.0 with 5 bits: (3,2); (4,2) has 6 bits
    w, _ = alloc.allocate(cost, bits, budget=3.0)
    assert w.tolist() == [3, 2]


def test_allocate_mutation_ignoring_budget_fails():
    cost = np.array([[10.0, 4.0, 1.0], [2.0, 1.5, 1.0], [6.0, 3.0, 2.0]])
    greedy = [int(np.argmin(r)) for r in cost]          # cheapest width per layer, no budget
    w, _ = alloc.allocate(cost, [2, 3, 4], budget=3.0)
    assert w.tolist() != [[2, 3, 4][j] for j in greedy]
