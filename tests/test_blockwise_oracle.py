"""Pins of the block-wise ("Lat.") layer of the oracle (CPU only).

The oracle computes y[b][n] = sum_i sum_c ldexp(sum_j s_i[n][8c+j] x[b][8c+j],
E[i][n // row_block][c]): one power-of-two factor per plane, block of rows and
8-column key (Sec. 4.2, block-wise scaling factors; Eq. 2).  Pinned against: a
hand-worked example; the row-wise layer of the oracle (another C function)
with groups of 8 and the block exponents repeated over the rows of a block,
which must agree bit for bit; a BLAS dense reconstruction; exact rationals.
Planted mistakes in a numpy restatement fail the dense pin.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "blockwise_hand.json")


def per_row(blk_exps, N, row_block):
    return np.repeat(blk_exps, row_block, axis=1)[:, :N]


def dense(signs, blk_exps, row_block):
    q, N, K = signs.shape
    f = np.ldexp(1.0, np.repeat(per_row(blk_exps, N, row_block).astype(np.int64), 8, axis=2))
    return (signs.astype(np.float64) * f).sum(0)


def test_hand_example():
    g = json.load(open(GOLDEN))
    y, a = oracle.shiftadd_gemm_blockwise(np.array(g["x"], np.float64),
                                          np.array(g["signs"], np.int8),
                                          np.array(g["blk_exps"], np.int8), g["row_block"])
    assert y.tolist() == g["y"]
    assert a.tolist() == g["absterm"]


@pytest.mark.parametrize("q,N,K,B,rb", [(1, 9, 64, 1, 2), (3, 100, 256, 2, 16), (2, 64, 1024, 3, 8),
                                        (4, 33, 128, 1, 33)])
def test_reduces_to_row_wise_groups_of_eight(q, N, K, B, rb):
    c = workloads.blockwise_case(q, N, K, B, rb, seed=2)
    y, a = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb)
    y_row, a_row = oracle.shiftadd_gemm(c["x"], c["signs"], per_row(c["blk_exps"], N, rb), 8)
    assert np.array_equal(y, y_row) and np.array_equal(a, a_row)


@pytest.mark.parametrize("q,N,K,B,rb", [(2, 40, 128, 2, 5), (3, 128, 512, 4, 16)])
def test_dense_reconstruction(q, N, K, B, rb):
    c = workloads.blockwise_case(q, N, K, B, rb, seed=3)
    y, a = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb)
    y_d = c["x"].astype(np.float64) @ dense(c["signs"], c["blk_exps"], rb).T
    assert np.abs(y - y_d).max() <= 1e-12 * a.max()


def test_exact_rational_brute_force():
    rb = 3
    c = workloads.blockwise_case(2, 7, 16, 2, rb, seed=4, exp_range=(-4, 4))
    y, _ = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb)
    for b in range(2):
        for n in range(7):
            exact = sum(Fraction(int(c["signs"][i, n, k])) * Fraction(float(c["x"][b, k]))
                        * Fraction(2) ** int(c["blk_exps"][i, n // rb, k // 8])
                        for i in range(2) for k in range(16))
            assert abs(Fraction(y[b, n]) - exact) <= Fraction(2) ** -50 * (abs(exact) + 1)


def _restated(x, signs, blk_exps, rb, mistake):
    q, N, K = signs.shape
    e = blk_exps.astype(np.int64)
    NB = e.shape[1]
    if mistake == "row_block_modulo":      # block index n % NB instead of n // rb
        er = e[:, np.arange(N) % NB]
    elif mistake == "sixteen_columns":     # a factor per 16 columns
        er = per_row(e, N, rb)[:, :, np.arange(K // 8) // 2]
    elif mistake == "negated":
        er = -per_row(e, N, rb)
    else:
        er = per_row(e, N, rb)
    f = np.ldexp(1.0, np.repeat(er, 8, axis=2))
    if mistake == "dropped_plane":
        f[-1] = 0.0
    W = (signs.astype(np.float64) * f).sum(0)
    return x.astype(np.float64) @ W.T


@pytest.mark.parametrize("mistake", ["row_block_modulo", "sixteen_columns", "negated",
                                     "dropped_plane"])
def test_planted_mistakes_fail_the_dense_pin(mistake):
    rb = 8
    c = workloads.blockwise_case(3, 48, 256, 2, rb, seed=6)
    y, a = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb)
    good = _restated(c["x"], c["signs"], c["blk_exps"], rb, None)
    bad = _restated(c["x"], c["signs"], c["blk_exps"], rb, mistake)
    assert np.abs(y - good).max() <= 1e-12 * a.max()
    assert np.abs(y - bad).max() > 1e-3 * a.max()
