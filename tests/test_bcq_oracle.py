"""Pins for the quantizer oracle (oracle/bcq.py), each against something other
than the oracle itself:

* a hand-worked segment (tests/golden/bcq_hand.json), including a BS tie;
* the q = 1 closed form of Sec. 3 (b = sign(w), alpha = w^T b / n);
* the Pythagorean identity of a greedy step: ||r_i||^2 = ||r_{i-1}||^2 - G alpha_i^2;
* an independent least-squares solver (numpy.linalg.lstsq) for the LS step,
  and the normal equations on rank-deficient codes;
* log2 bounds for the PoT rounding;
* brute force over all 2^q codes (itertools) for the BS step;
* exact recovery of weights that already have the format (powers of two times
  +-1 patterns);
* the layer format: reconstruct(signs, exps) equals sum_i PoT(alpha_i) b_i;
* mutations: copies of the quantizer with one plausible mistake fail a pin.
"""
import itertools
from fractions import Fraction
import json
import os

import numpy as np
import pytest

import workloads
from oracle import bcq

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _hand():
    with open(os.path.join(GOLDEN, "bcq_hand.json")) as f:
        return json.load(f)


def _rand_w(seed, S, G, scale=0.02):
    return np.random.default_rng(seed).normal(0, scale, (S, G))


# ----------------------------------------------------------------------------- hand example

def test_hand_segment_greedy_pot_and_cycle():
    h = _hand()["segment"]
    w = np.array([h["w"]], np.float64)
    B, A = bcq.greedy(w, h["q"])
    assert B[0].tolist() == h["greedy_codes"]
    assert A[0].tolist() == h["greedy_alphas"]
    sgn, P = bcq.pot(A)
    assert P[0].tolist() == h["pot_exponents"] and (sgn == 1).all()
    assert bcq.least_squares(B, w)[0].tolist() == h["cycle1_alphas_ls"]
    B1, pa = bcq.quantize_segments(w, h["q"], 1)
    assert B1[0].tolist() == h["cycle1_codes"]
    assert np.einsum("si,sig->sg", pa, B1)[0].tolist() == h["cycle1_reconstruction"]


def test_hand_zero_segment():
    h = _hand()["zero_segment"]
    w = np.array([h["w"]], np.float64)
    for cycles, key in ((0, "signs_no_cycles"), (2, "signs_after_cycles")):
        signs, exps = bcq.quantize(w, h["q"], 8, cycles)
        assert signs[:, 0, :].tolist() == h[key]
        assert exps[:, 0, 0].tolist() == h["exps"]


# ----------------------------------------------------------------------------- greedy

def test_q1_closed_form():
    w = _rand_w(1, 50, 128)
    B, A = bcq.greedy(w, 1)
    assert np.array_equal(B[:, 0], np.where(w >= 0, 1.0, -1.0))
    np.testing.assert_allclose(A[:, 0], np.abs(w).mean(axis=1), rtol=1e-14)


@pytest.mark.parametrize("q", [2, 3, 8])
def test_greedy_pythagoras(q):
    """alpha_i b_i is the orthogonal projection of r_{i-1} on b_i."""
    w = _rand_w(2, 40, 64)
    B, A = bcq.greedy(w, q)
    r = w.copy()
    for i in range(q):
        prev = np.square(r).sum(axis=1)
        r = r - A[:, i:i + 1] * B[:, i]
        now = np.square(r).sum(axis=1)
        np.testing.assert_allclose(now, prev - w.shape[1] * A[:, i] ** 2, rtol=1e-9, atol=1e-18)
        assert (A[:, i] >= 0).all()


# ----------------------------------------------------------------------------- LS

def test_least_squares_matches_lstsq():
    w = _rand_w(3, 30, 128)
    for q in (1, 2, 3, 4, 8):
        B, _ = bcq.greedy(w, q)
        A = bcq.least_squares(B, w)
        for s in range(w.shape[0]):
            ref = np.linalg.lstsq(B[s].T, w[s], rcond=None)[0]
            np.testing.assert_allclose(A[s], ref, rtol=1e-9, atol=1e-15)


def test_least_squares_rank_deficient():
    """Dependent code vectors get alpha = 0; the kept ones solve the normal
    equations, so the residual equals the least-squares residual."""
    rng = np.random.default_rng(4)
    G = 64
    w = rng.normal(size=(1, G))
    b1 = np.where(rng.random(G) < 0.5, 1.0, -1.0)
    b3 = np.where(rng.random(G) < 0.5, 1.0, -1.0)
    B = np.stack([b1, -b1, b3])[None]               # b2 = -b1
    A = bcq.least_squares(B, w)
    assert A[0, 1] == 0.0
    fit = np.einsum("si,sig->sg", A, B)
    ref = np.linalg.lstsq(B[0].T, w[0], rcond=None)[0]
    np.testing.assert_allclose(fit[0], B[0].T @ ref, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(B[0] @ (w[0] - fit[0]), 0, atol=1e-9)


# ----------------------------------------------------------------------------- PoT

def test_pot_rounds_in_log_domain():
    rng = np.random.default_rng(5)
    a = rng.normal(size=2000) * np.exp(rng.uniform(-20, 20, 2000))
    sgn, P = bcq.pot(a)
    assert np.array_equal(sgn, np.where(a < 0, -1.0, 1.0))
    assert (np.abs(np.log2(np.abs(a)) - P) <= 0.5 + 1e-12).all()
    k = np.arange(-40, 41)
    assert np.array_equal(bcq.pot(np.ldexp(1.0, k))[1], k)
    assert np.array_equal(bcq.pot(-np.ldexp(1.0, k))[1], k)
    assert bcq.pot(np.array([0.0]))[1][0] == -128
    assert bcq.pot(np.array([2.0 ** 200]))[1][0] == 127


# ----------------------------------------------------------------------------- BS

@pytest.mark.parametrize("q", [1, 2, 3, 5])
def test_binary_search_is_brute_force_nearest(q):
    rng = np.random.default_rng(6 + q)
    S, G = 6, 32
    w = rng.normal(size=(S, G))
    a = bcq.pot_values(rng.normal(size=(S, q)))
    B = bcq.binary_search(a, w)
    for s in range(S):
        codes = list(itertools.product((-1.0, 1.0), repeat=q))
        vals = [float(np.dot(c, a[s])) for c in codes]
        for g in range(G):
            dists = [abs(w[s, g] - v) for v in vals]
            got = float(np.dot(B[s, :, g], a[s]))
            assert abs(w[s, g] - got) == min(dists)


def test_binary_search_tie_goes_to_smaller_code():
    a = np.array([[2.0, 1.0]])
    w = np.array([[-2.0, 0.0, 2.0]])
    B = bcq.binary_search(a, w)
    # -2: codes 0 (-3) and 2 (-1) tie -> code 0; 0: codes 1 (+1) and 2 (-1) tie -> code 1;
    # 2: codes 1 (+1) and 3 (+3) tie -> code 1
    assert B[0, :, 0].tolist() == [-1.0, -1.0]
    assert B[0, :, 1].tolist() == [1.0, -1.0]
    assert B[0, :, 2].tolist() == [1.0, -1.0]


def test_each_step_does_not_increase_the_error():
    """LS minimises over alpha for fixed codes; BS minimises over codes for fixed
    alpha (the PoT rounding between them may increase it)."""
    w = _rand_w(7, 30, 128)
    for q in (2, 3):
        B, A = bcq.greedy(w, q)
        err = lambda A_, B_: np.square(w - np.einsum("si,sig->sg", A_, B_)).sum(axis=1)  # noqa
        A_ls = bcq.least_squares(B, w)
        assert (err(A_ls, B) <= err(A, B) * (1 + 1e-12)).all()
        pa = bcq.pot_values(A_ls)
        B_bs = bcq.binary_search(pa, w)
        assert (err(pa, B_bs) <= err(pa, B) * (1 + 1e-12) + 1e-30).all()


# ----------------------------------------------------------------------------- whole quantizer

@pytest.mark.parametrize("q", [1, 2])
def test_exact_recovery_of_formatted_weights(q):
    """A weight that already is sum_i 2^P_i b_i with dominant leading terms is
    recovered exactly (zero error) after one cycle."""
    rng = np.random.default_rng(8)
    N, K, G = 16, 256, 128
    P = rng.integers(-9, -5, (N, K // G))
    W = np.zeros((N, K))
    for i in range(q):
        b = np.where(rng.random((N, K)) < 0.5, 1.0, -1.0)
        W += np.repeat(np.ldexp(1.0, P - 2 * i), G, axis=1) * b
    signs, exps = bcq.quantize(W, q, G, cycles=1)
    assert np.array_equal(bcq.reconstruct(signs, exps, G), W)


def test_format_and_sign_folding():
    rng = np.random.default_rng(9)
    N, K, G, q = 8, 384, 128, 3
    W = rng.normal(0, 0.02, (N, K))
    B, pa = bcq.quantize_segments(bcq.segments(W, G), q, 2)
    signs, exps = bcq.quantize(W, q, G, 2)
    assert set(np.unique(signs)) <= {-1, 1}
    direct = np.einsum("si,sig->sg", pa, B).reshape(N, K)
    assert np.array_equal(bcq.reconstruct(signs, exps, G), direct)


def test_quantization_error_is_sane():
    """3-bit BCQ with one power-of-two term per scale on Gaussian weights: the
    alternating cycles do not end worse than the greedy start, and the relative
    L2 error stays in the range the format allows (about 0.26 here)."""
    W = _rand_w(10, 64, 1024)
    rel = []
    for cycles in (0, 1, 3):
        signs, exps = bcq.quantize(W, 3, 128, cycles)
        rel.append(np.linalg.norm(bcq.reconstruct(signs, exps, 128) - W) / np.linalg.norm(W))
    assert rel[2] <= rel[1] <= rel[0] < 0.3


# ----------------------------------------------------------------------------- mutations

def _mut_greedy_no_residual(w, q):
    S, G = w.shape
    B = np.empty((S, q, G)); A = np.empty((S, q))
    for i in range(q):                               # forgets to update the residual
        B[:, i] = bcq.sign_pm1(w); A[:, i] = (w * B[:, i]).sum(axis=1) / G
    return B, A


def _mut_greedy_sum_not_mean(w, q):
    B, A = bcq.greedy(w, q)
    return B, A * w.shape[1]


def _mut_pot_floor(alpha):
    sgn, P = bcq.pot(alpha)
    m, E = np.frexp(np.abs(alpha))
    return sgn, np.where(np.abs(alpha) == 0, -128, E - 1)   # floor, not round


def test_mutations_fail_pins(monkeypatch):
    h = _hand()["segment"]
    w = np.array([h["w"]], np.float64)
    assert _mut_greedy_no_residual(w, 2)[0].tolist() != [h["greedy_codes"]]
    assert _mut_greedy_sum_not_mean(w, 2)[1][0].tolist() != h["greedy_alphas"]
    assert _mut_pot_floor(np.array(h["greedy_alphas"]))[1].tolist() != h["pot_exponents"]
    # a BS that breaks ties toward the larger code picks code 2, not the
    # fixture's code 0, for w = -2 with scales (2, 1)
    vals = bcq.code_values(np.array([[2.0, 1.0]]))[0]
    dist = np.abs(-2.0 - vals)
    assert int(np.flatnonzero(dist == dist.min())[-1]) == 2


# ----------------------------------------------------------- additive PoT (Eq. 2, several terms)

def test_pot_terms_hand_example():
    # alpha = 0.8: round(log2 0.8) = 0 -> +1; residual -0.2 -> round(log2 0.2) = -2 -> -1/4;
    # residual 0.05 -> round(log2 0.05) = -4 -> +1/16; value 1 - 1/4 + 1/16 = 0.8125
    v, sg, P = bcq.pot_terms(np.array([0.8]), 3)
    assert v.tolist() == [0.8125]
    assert sg.ravel().tolist() == [1, -1, 1] and P.ravel().tolist() == [0, -2, -4]


def test_pot_terms_one_term_is_pot():
    a = np.random.default_rng(1).standard_normal(1000) * 0.03
    v, sg, P = bcq.pot_terms(a, 1)
    s1, P1 = bcq.pot(a)
    assert np.array_equal(v, bcq.pot_values(a)) and np.array_equal(P[0], P1)
    assert np.array_equal(sg[0], s1)


def test_pot_terms_residuals_are_exact_and_contract():
    """Each term is within a factor sqrt(2) of its residual, so the subtraction
    is exact (Sterbenz) and the residual shrinks by at least sqrt(2) - 1."""
    a = np.random.default_rng(2).standard_normal(2000) * 0.05
    r = a.copy()
    for T in range(1, 5):
        v, sg, P = bcq.pot_terms(a, T)
        r_new = a - v
        for x, vv in zip(a[:50], v[:50]):
            assert Fraction(float(x)) - Fraction(float(vv)) == Fraction(float(x - vv))
        assert (np.abs(r_new) <= (np.sqrt(2) - 1) * np.abs(r) + 1e-300).all()
        r = r_new


def test_pot_terms_zero_and_powers_of_two():
    v, sg, P = bcq.pot_terms(np.array([0.0, 0.25, -4.0]), 3)
    assert v.tolist() == [0.0, 0.25, -4.0]
    assert sg[:, 0].tolist() == [0, 0, 0]
    assert sg[:, 1].tolist() == [1, 0, 0] and sg[:, 2].tolist() == [-1, 0, 0]


def test_quantize_terms_one_term_is_quantize():
    w = workloads.fp_weights(16, 512, seed=5)
    s1, e1 = bcq.quantize(w, 3, 128, 2)
    s, e, t = bcq.quantize_terms(w, 3, 128, 2, 1)
    assert np.array_equal(s, s1) and np.array_equal(e[..., 0], e1)
    assert set(np.unique(t)) <= {0, 1}


def test_quantize_terms_format_and_error():
    w = workloads.fp_weights(32, 512, seed=6)
    errs = []
    for T in (1, 2, 3):
        s, e, t = bcq.quantize_terms(w, 3, 128, 2, T)
        assert (t[..., 0] >= 0).all() and set(np.unique(t)) <= {-1, 0, 1}
        B, pa = bcq.quantize_segments(bcq.segments(w, 128), 3, 2, terms=T)
        direct = np.einsum("si,sig->sg", pa, B).reshape(w.shape)
        assert np.array_equal(bcq.reconstruct_terms(s, e, t, 128), direct)
        errs.append(np.linalg.norm(direct - w) / np.linalg.norm(w))
    assert errs[1] < errs[0] and errs[2] <= errs[1] * 1.01


def test_pot_terms_mutation_without_residual_fails(monkeypatch):
    def no_residual(alpha, terms):      # every term rounds alpha itself
        v = np.zeros_like(alpha)
        for _ in range(terms):
            v = v + bcq.pot_values(alpha)
        return v, None, None
    monkeypatch.setattr(bcq, "pot_terms", no_residual)
    with pytest.raises(AssertionError):
        test_pot_terms_hand_example()
