"""Pins of the layer with additive power-of-two factors (Eq. 2 with T terms) of
the oracle (CPU only): a hand example; bit-for-bit agreement with the
single-term row-wise layer (another C function) for T = 1; a sign-0 term is the
same as no term; two equal terms equal one term of twice the size; a BLAS
dense reconstruction; exact rationals.  Planted mistakes fail the dense pin.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "terms_hand.json")


def dense(signs, exps, term_signs, G):
    f = (term_signs.astype(np.float64) * np.ldexp(1.0, exps.astype(np.int64))).sum(-1)  # [q][N][NG]
    return (signs.astype(np.float64) * np.repeat(f, G, axis=2)).sum(0)


def test_hand_example():
    g = json.load(open(GOLDEN))
    y, a = oracle.shiftadd_gemm_terms(np.array(g["x"], np.float64), np.array(g["signs"], np.int8),
                                      np.array(g["exps"], np.int8),
                                      np.array(g["term_signs"], np.int8), g["G"])
    assert y.tolist() == g["y"] and a.tolist() == g["absterm"]


@pytest.mark.parametrize("q,N,K,G,B", [(1, 9, 64, 8, 1), (3, 50, 512, 128, 2), (2, 33, 384, 384, 3)])
def test_one_term_is_the_row_wise_layer(q, N, K, G, B):
    c = workloads.terms_case(q, N, K, G, B, 1, seed=2)
    y, a = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], G)
    y_row, a_row = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"][..., 0], G)
    assert np.array_equal(y, y_row) and np.array_equal(a, a_row)


def test_sign_zero_term_is_no_term():
    c = workloads.terms_case(3, 40, 256, 128, 2, 3, seed=3)
    ts = c["term_signs"].copy()
    ts[..., 2] = 0
    y, a = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], ts, 128)
    y2, a2 = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"][..., :2].copy(),
                                        ts[..., :2].copy(), 128)
    assert np.array_equal(y, y2) and np.array_equal(a, a2)


def test_two_equal_terms_are_one_doubled_term():
    c = workloads.terms_case(2, 40, 256, 128, 2, 1, seed=4)
    e2 = np.concatenate([c["exps"], c["exps"]], axis=-1)
    s2 = np.ones_like(e2)
    y, a = oracle.shiftadd_gemm_terms(c["x"], c["signs"], e2, s2, 128)
    y1, a1 = oracle.shiftadd_gemm(c["x"], c["signs"], (c["exps"][..., 0] + 1).astype(np.int8), 128)
    assert np.abs(y - y1).max() <= 1e-12 * a.max() and np.abs(a - a1).max() <= 1e-12 * a.max()


@pytest.mark.parametrize("T", [2, 3, 4])
def test_dense_reconstruction(T):
    c = workloads.terms_case(3, 64, 512, 128, 3, T, seed=5)
    y, a = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], 128)
    y_d = c["x"].astype(np.float64) @ dense(c["signs"], c["exps"], c["term_signs"], 128).T
    assert np.abs(y - y_d).max() <= 1e-12 * a.max()


def test_exact_rational_brute_force():
    c = workloads.terms_case(2, 5, 32, 8, 2, 3, seed=6, exp_range=(-3, 3))
    y, _ = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], 8)
    for b in range(2):
        for n in range(5):
            exact = Fraction(0)
            for i in range(2):
                for k in range(32):
                    f = sum(Fraction(int(c["term_signs"][i, n, k // 8, t]))
                            * Fraction(2) ** int(c["exps"][i, n, k // 8, t]) for t in range(3))
                    exact += Fraction(int(c["signs"][i, n, k])) * Fraction(float(c["x"][b, k])) * f
            assert abs(Fraction(y[b, n]) - exact) <= Fraction(2) ** -50 * (abs(exact) + 1)


@pytest.mark.parametrize("mistake", ["signs_ignored", "first_term_only", "terms_swapped_planes"])
def test_planted_mistakes_fail_the_dense_pin(mistake):
    c = workloads.terms_case(3, 48, 256, 128, 2, 3, seed=7)
    y, a = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], 128)
    e, ts = c["exps"].copy(), c["term_signs"].copy()
    if mistake == "signs_ignored":
        ts = np.abs(ts)
    elif mistake == "first_term_only":
        ts[..., 1:] = 0
    else:
        e[..., 1] = e[::-1, ..., 1]
    bad = c["x"].astype(np.float64) @ dense(c["signs"], e, ts, 128).T
    assert np.abs(y - bad).max() > 1e-3 * a.max()
