"""CPU oracle for the automated mixed-bit allocation of ShiftAddLLM (fp64,
numpy).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  The product path
(``paper_2406_05981_amd``) never imports it and shares no code with it.

What it computes (Sec. 4.3; parity is pinned by ``tests/test_alloc_oracle.py``):

* ``criterion`` -- Eq. 3 for one layer with weights W [N][K] and calibration
  activations X [K][T] (one column per token):
  IS = W / diag(cholesky((X X^T)^{-1})) (each column k of W divided by the k-th
  diagonal entry of the Cholesky factor of the inverse), C = ||IS||_F STD(IS)^2.
* ``fit_per_bit`` -- the least-squares polynomial fits that turn the criterion
  into a per-bit estimate: for each bit width b, a polynomial p_b of the given
  degree is fitted to the pairs (C_i, E_{i,b}) of measured errors, and
  C_{i,b} = p_b(C_i).
* ``allocate`` -- Eq. 4: one bit width per layer minimising sum_i C_{i,b_i}
  under sum_i b_i <= B L, by exhaustive enumeration (small L only).

Readings where the paper is silent:

* X X^T is damped before the inverse: H = X X^T + damp * mean(diag(X X^T)) I,
  damp = 0.01 by default (the usual convention of the OBC/OPTQ line of work the
  criterion comes from); without it a rank-deficient calibration set has no
  inverse.
* cholesky is the lower factor L (A = L L^T); the upper factor of the same
  matrix has the same diagonal.
* STD is the population standard deviation over all N K entries of IS.
* The budget B L is a bound on the total bits, B the average bits per layer.
* Ties in Eq. 4 (equal objective): fewer total bits first, then the
  lexicographically smallest bit vector (layer 0 first).  The objective of an
  assignment is summed over the layers in order, from layer 0.
"""
from __future__ import annotations

import itertools
from typing import Sequence, Tuple

import numpy as np


def gram(x: np.ndarray) -> np.ndarray:
    """X X^T in fp64 for X [K][T]."""
    x = np.asarray(x, np.float64)
    return x @ x.T


def damped(H: np.ndarray, damp: float) -> np.ndarray:
    return H + damp * np.mean(np.diag(H)) * np.eye(H.shape[0])


def cholesky_diag_of_inverse(H: np.ndarray) -> np.ndarray:
    """diag(cholesky(H^{-1})), literally: invert, then factor."""
    return np.diag(np.linalg.cholesky(np.linalg.inv(H)))


def importance(w: np.ndarray, x: np.ndarray, damp: float = 0.01) -> np.ndarray:
    """IS = W / diag(cholesky((X X^T + damping)^{-1})), column by column."""
    d = cholesky_diag_of_inverse(damped(gram(x), damp))
    return np.asarray(w, np.float64) / d[None, :]


def criterion(w: np.ndarray, x: np.ndarray, damp: float = 0.01) -> float:
    """Eq. 3: C = ||IS||_F * STD(IS)^2."""
    IS = importance(w, x, damp)
    return float(np.linalg.norm(IS) * np.std(IS) ** 2)


def fit_per_bit(c: Sequence[float], errors: np.ndarray, degree: int = 1) -> np.ndarray:
    """Least-squares polynomial fits: for each bit width (column of errors
    [L][nb]) fit E_b ~ p_b(C); returns C_{i,b} = p_b(C_i), [L][nb]."""
    c = np.asarray(c, np.float64)
    errors = np.asarray(errors, np.float64)
    out = np.empty_like(errors)
    for b in range(errors.shape[1]):
        coef = np.polyfit(c, errors[:, b], degree)
        out[:, b] = np.polyval(coef, c)
    return out


def allocate(cost: np.ndarray, bits: Sequence[int], budget: float) -> Tuple[np.ndarray, float]:
    """Eq. 4 by enumeration: the bit width per layer (one-hot beta written as
    the chosen width) minimising sum_i cost[i][choice] under
    sum_i bits[choice] <= budget * L.  Returns (widths [L], objective)."""
    cost = np.asarray(cost, np.float64)
    L, nb = cost.shape
    cap = budget * L
    best = None
    for choice in itertools.product(range(nb), repeat=L):
        total_bits = sum(bits[j] for j in choice)
        if total_bits > cap:
            continue
        obj = 0.0
        for i, j in enumerate(choice):
            obj = obj + cost[i, j]
        key = (obj, total_bits, tuple(bits[j] for j in choice))
        if best is None or key < best[0]:
            best = (key, choice)
    if best is None:
        raise ValueError("no assignment fits the budget")
    widths = np.array([bits[j] for j in best[1]], dtype=np.int64)
    return widths, best[0][0]
