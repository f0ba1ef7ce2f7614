"""Pins of the column-wise ("Acc.") layer of the oracle (CPU only).

The oracle computes y[b][n] = sum_i sum_k s_i[n][k] ldexp(x[b][k], e[i][k]) with
one power-of-two factor per plane and weight column (Sec. 4.2, column-wise
scaling factors; Eq. 2 for the power of two).  It is pinned here against: a
hand-worked example; the row-wise layer of the oracle (a different C function)
when every column of a plane has the same exponent (then the factor leaves the
sum, exactly); a dense reconstruction of W_q multiplied by BLAS; exact rational
arithmetic on tiny shapes; invariance under a joint permutation of the columns.
Plausible mistakes planted in a numpy restatement are rejected by the dense pin.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "colwise_hand.json")


def dense(signs, col_exps):
    return (signs.astype(np.float64) * np.ldexp(1.0, col_exps.astype(np.int64))[:, None, :]).sum(0)


def test_hand_example():
    g = json.load(open(GOLDEN))
    y, a = oracle.shiftadd_gemm_colwise(np.array(g["x"], np.float64), np.array(g["signs"], np.int8),
                                        np.array(g["col_exps"], np.int8))
    assert y.tolist() == g["y"]
    assert a.tolist() == g["absterm"]


@pytest.mark.parametrize("q,N,K,B", [(1, 9, 64, 1), (3, 33, 256, 2), (4, 17, 1024, 3)])
def test_constant_columns_reduce_to_row_wise_layer(q, N, K, B):
    c = workloads.colwise_case(q, N, K, B, seed=2)
    e = c["col_exps"][:, :1].repeat(K, axis=1)  # one exponent per plane
    y, a = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], e)
    exps = np.broadcast_to(e[:, None, :1], (q, N, 1)).copy()
    y_row, a_row = oracle.shiftadd_gemm(c["x"], c["signs"], exps, K)
    assert np.array_equal(y, y_row) and np.array_equal(a, a_row)


@pytest.mark.parametrize("q,N,K,B", [(2, 40, 128, 2), (3, 64, 512, 4)])
def test_dense_reconstruction(q, N, K, B):
    c = workloads.colwise_case(q, N, K, B, seed=3)
    y, a = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"])
    y_d = c["x"].astype(np.float64) @ dense(c["signs"], c["col_exps"]).T
    assert np.abs(y - y_d).max() <= 1e-12 * a.max()
    a_d = np.abs(c["x"].astype(np.float64)) @ np.abs(dense(np.ones_like(c["signs"]), c["col_exps"])).T
    assert np.abs(a - a_d).max() <= 1e-12 * a.max()


def test_exact_rational_brute_force():
    c = workloads.colwise_case(3, 5, 16, 2, seed=4, exp_range=(-4, 4))
    y, _ = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"])
    for b in range(2):
        for n in range(5):
            exact = sum(Fraction(int(c["signs"][i, n, k])) * Fraction(float(c["x"][b, k]))
                        * Fraction(2) ** int(c["col_exps"][i, k])
                        for i in range(3) for k in range(16))
            assert abs(Fraction(y[b, n]) - exact) <= Fraction(2) ** -50 * (abs(exact) + 1)


def test_joint_column_permutation():
    c = workloads.colwise_case(3, 20, 256, 2, seed=5)
    perm = np.random.default_rng(0).permutation(256)
    y, a = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"])
    y_p, _ = oracle.shiftadd_gemm_colwise(c["x"][:, perm], c["signs"][:, :, perm],
                                          c["col_exps"][:, perm])
    assert np.abs(y - y_p).max() <= 1e-12 * a.max()


def _restated(x, signs, col_exps, mistake):
    s = signs.astype(np.float64)
    e = col_exps.astype(np.int64)
    q, N, K = signs.shape
    if mistake == "row_axis":           # factor indexed by output row
        f = np.ldexp(1.0, e[:, :N])[:, :, None] * np.ones((1, 1, K))
    elif mistake == "negated_exponent":
        f = np.ldexp(1.0, -e)[:, None, :] * np.ones((1, N, 1))
    elif mistake == "dropped_plane":
        f = np.ldexp(1.0, e)[:, None, :] * np.ones((1, N, 1))
        f[-1] = 0.0
    elif mistake == "shared_first_plane_exponent":
        f = np.ldexp(1.0, e[:1])[:, None, :] * np.ones((q, N, 1))
    else:
        f = np.ldexp(1.0, e)[:, None, :] * np.ones((1, N, 1))
    W = (s * f).sum(0)
    return x.astype(np.float64) @ W.T


@pytest.mark.parametrize("mistake", ["row_axis", "negated_exponent", "dropped_plane",
                                     "shared_first_plane_exponent"])
def test_planted_mistakes_fail_the_dense_pin(mistake):
    c = workloads.colwise_case(3, 48, 128, 2, seed=6)
    y, a = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"])
    good = _restated(c["x"], c["signs"], c["col_exps"], None)
    bad = _restated(c["x"], c["signs"], c["col_exps"], mistake)
    assert np.abs(y - good).max() <= 1e-12 * a.max()
    assert np.abs(y - bad).max() > 1e-3 * a.max()
