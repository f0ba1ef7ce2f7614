"""Pins for the CPU oracle: each checks it against something other than itself.

* hand-worked fixtures (tests/golden/hand_examples.json),
* closed forms and invariants of the table of Sec. 4.1,
* an independent library implementation (numpy packbits) of the key packing,
* a dense route (reconstruct W_q = sum_i 2^e b_i and multiply with BLAS),
* exact rational brute force on tiny inputs,
* exact invariants of the layer (power-of-two shift, linearity, complement,
  plane permutation, the +-1 matvec special case),
* mutation checks: copies of the definition with one plausible mistake each must
  fail at least one of the pins above.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _hand():
    with open(os.path.join(GOLDEN, "hand_examples.json")) as f:
        return json.load(f)


# ----------------------------------------------------------------------------- packing

def test_pack_fixed_patterns(oracle_mod):
    q, N, K = 2, 3, 64
    plus = np.ones((q, N, K), np.int8)
    assert (oracle_mod.pack(plus) == 0xFF).all()
    assert (oracle_mod.pack(-plus) == 0x00).all()
    # zero counts as -1
    assert (oracle_mod.pack(np.zeros((q, N, K), np.int8)) == 0x00).all()
    for j in range(8):
        s = -np.ones((q, N, K), np.int8)
        s[..., j::8] = 1
        assert (oracle_mod.pack(s) == (1 << j)).all(), j


def test_pack_matches_numpy_packbits(oracle_mod):
    c = workloads.random_case(3, 37, 200, 8, 1, seed=3)
    ref = np.packbits(c["signs"] > 0, axis=-1, bitorder="little")
    assert np.array_equal(oracle_mod.pack(c["signs"]), ref)


def test_unpack_roundtrip(oracle_mod):
    c = workloads.random_case(4, 19, 128, 8, 1, seed=4)
    p = oracle_mod.pack(c["signs"])
    assert np.array_equal(oracle_mod.unpack(p, 128), c["signs"])
    rng = np.random.default_rng(0)
    raw = rng.integers(0, 256, (2, 5, 7), dtype=np.uint8)
    assert np.array_equal(oracle_mod.pack(oracle_mod.unpack(raw, 56)), raw)


def test_pack_hand_example(oracle_mod):
    h = _hand()["layer"]
    s = np.array(h["signs"], np.int8)
    assert oracle_mod.pack(s).tolist() == h["packed"]


# ----------------------------------------------------------------------------- table

def test_lut_hand_example(oracle_mod):
    h = _hand()["lut_chunk"]
    x = np.array([h["x"]], np.float16)
    t = oracle_mod.lut(x)[0, 0]
    for key, val in h["entries"].items():
        assert t[int(key)] == val, key


def _bits256():
    return ((np.arange(256)[:, None] >> np.arange(8)[None, :]) & 1).astype(np.float64)


@pytest.mark.parametrize("seed", [0, 1])
def test_lut_closed_form_exact(oracle_mod, seed):
    """lut[m] = 2 * (sum of x_j over set bits j of m) - (sum of x)."""
    c = workloads.random_case(1, 1, 96, 8, 3, seed=seed, outlier_fraction=0.05)
    x = c["x"].astype(np.float64)
    t = oracle_mod.lut(c["x"])
    xc = x.reshape(3, 12, 8)
    closed = 2.0 * np.einsum("mj,bcj->bcm", _bits256(), xc) - xc.sum(-1)[..., None]
    assert np.array_equal(t, closed)


def test_lut_invariants(oracle_mod):
    c = workloads.random_case(1, 1, 64, 8, 2, seed=5, outlier_fraction=0.1)
    x = c["x"].astype(np.float64).reshape(2, 8, 8)
    t = oracle_mod.lut(c["x"])
    s = x.sum(-1)
    assert np.array_equal(t[..., 0xFF], s)
    assert np.array_equal(t[..., 0x00], -s)
    m = np.arange(256)
    assert np.array_equal(t[..., 255 - m], -t[..., m])  # LUT[~m] = -LUT[m]
    for j in range(8):
        lo = m[(m >> j) & 1 == 0]
        assert np.array_equal(t[..., lo | (1 << j)] - t[..., lo], 2.0 * np.repeat(x[..., j:j + 1], lo.size, -1))


def test_query_add_identity_all_keys(oracle_mod):
    """With q=1, e=0 and G=8, the layer over an 8-column input whose row n is the
    key n returns the table itself: query + add of one key is one table entry."""
    keys = np.arange(256, dtype=np.uint8).reshape(1, 256, 1)
    signs = oracle_mod.unpack(keys, 8)
    exps = np.zeros((1, 256, 1), np.int8)
    c = workloads.random_case(1, 1, 8, 8, 2, seed=9)
    y, _ = oracle_mod.shiftadd_gemm(c["x"], signs, exps, 8)
    t = oracle_mod.lut(c["x"])
    assert np.array_equal(y, t[:, 0, :])


# ----------------------------------------------------------------------------- the layer

def _dense(case):
    """Independent route: W_q = sum_i 2^e_i * s_i (exact in fp64), y = x W_q^T via BLAS."""
    s, e, G = case["signs"].astype(np.float64), case["exps"], case["G"]
    scale = np.ldexp(1.0, np.repeat(e.astype(np.int64), G, axis=2))
    W = (scale * s).sum(0)
    Wabs = scale.sum(0)
    x = case["x"].astype(np.float64)
    return x @ W.T, np.abs(x) @ Wabs.T


def test_layer_hand_example(oracle_mod):
    h = _hand()["layer"]
    y, a = oracle_mod.shiftadd_gemm(np.array(h["x"], np.float16), np.array(h["signs"], np.int8),
                                    np.array(h["exps"], np.int8), h["G"])
    assert y.tolist() == h["y"] and a.tolist() == h["absterm"]


DENSE_CASES = [
    (3, 64, 256, 128, 1), (2, 37, 384, 128, 3), (4, 5, 64, 8, 2), (1, 1, 8, 8, 1),
    (8, 9, 128, 16, 2), (3, 16, 768, 768, 1), (2, 33, 96, 24, 4),
]


@pytest.mark.parametrize("q,N,K,G,B", DENSE_CASES)
def test_dense_reconstruction(oracle_mod, q, N, K, G, B):
    c = workloads.random_case(q, N, K, G, B, seed=11, outlier_fraction=0.02)
    y, a = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"], G)
    yd, ad = _dense(c)
    assert np.all(np.abs(y - yd) <= 1e-12 * a)
    assert np.allclose(a, ad, rtol=1e-13, atol=0)


def test_dense_reconstruction_opt125m_full(oracle_mod):
    c = workloads.layer_inputs("opt125m_proj", 0, 1)
    y, a = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"], c["G"])
    yd, ad = _dense(c)
    assert np.all(np.abs(y - yd) <= 1e-12 * a)
    assert np.allclose(a, ad, rtol=1e-13, atol=0)


def _exact(case):
    """Exact rational value of every output (Python Fractions)."""
    s, e, G = case["signs"], case["exps"], case["G"]
    xs = [[Fraction(*float(v).as_integer_ratio()) for v in row] for row in case["x"].astype(np.float64)]
    q, N, K = s.shape
    out = []
    for b in range(len(xs)):
        ys, abss = [], []
        for n in range(N):
            tot = Fraction(0)
            ab = Fraction(0)
            for i in range(q):
                for k in range(K):
                    f = Fraction(2) ** int(e[i, n, k // G])
                    tot += int(s[i, n, k]) * xs[b][k] * f
                    ab += abs(xs[b][k]) * f
            ys.append(tot)
            abss.append(ab)
        out.append((ys, abss))
    return out


@pytest.mark.parametrize("q,N,K,G,B,lo,hi", [
    (1, 3, 8, 8, 1, -24, 15), (2, 8, 16, 8, 2, -24, 15), (3, 1, 64, 16, 3, -24, 15),
    (4, 3, 64, 64, 1, -24, 15), (2, 2, 256, 256, 2, -10, 10), (4, 256, 8, 8, 1, -24, 15),
])
def test_bruteforce_exact_rationals(oracle_mod, q, N, K, G, B, lo, hi):
    c = workloads.random_case(q, N, K, G, B, seed=21, exp_range=(lo, hi), outlier_fraction=0.1)
    y, a = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"], G)
    ex = _exact(c)
    for b in range(B):
        for n in range(N):
            yv, av = ex[b][0][n], ex[b][1][n]
            assert a[b, n] == float(av) or abs(Fraction(a[b, n]) - av) <= Fraction(2) ** -50 * av
            assert abs(Fraction(y[b, n]) - yv) <= Fraction(2) ** -50 * av


@pytest.mark.parametrize("delta", [-7, -1, 1, 5])
def test_exact_power_of_two_shift(oracle_mod, delta):
    c = workloads.random_case(3, 40, 512, 128, 2, seed=31, outlier_fraction=0.01)
    y, a = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128)
    y2, a2 = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"] + np.int8(delta), 128)
    assert np.array_equal(y2, np.ldexp(y, delta))
    assert np.array_equal(a2, np.ldexp(a, delta))


def test_linearity_and_odd_symmetry(oracle_mod):
    rng = np.random.default_rng(7)
    c = workloads.random_case(3, 24, 256, 32, 1, seed=41)
    x1 = rng.integers(-50, 50, (1, 256)).astype(np.float16)  # small integers: all sums exact
    x2 = rng.integers(-50, 50, (1, 256)).astype(np.float16)
    f = lambda x: oracle_mod.shiftadd_gemm(x, c["signs"], c["exps"], 32)[0]
    assert np.array_equal(f((x1.astype(np.float32) + x2).astype(np.float16)), f(x1) + f(x2))
    assert np.array_equal(f(-c["x"]), -f(c["x"]))


def test_complement_plane(oracle_mod):
    """Flipping every bit of plane i negates that plane's contribution."""
    rng = np.random.default_rng(8)
    c = workloads.random_case(3, 17, 192, 64, 2, seed=51)
    x = rng.integers(-20, 20, (2, 192)).astype(np.float16)
    y, _ = oracle_mod.shiftadd_gemm(x, c["signs"], c["exps"], 64)
    for i in range(3):
        s = c["signs"].copy()
        s[i] = -s[i]
        yf, _ = oracle_mod.shiftadd_gemm(x, s, c["exps"], 64)
        yi, _ = oracle_mod.shiftadd_gemm(x, c["signs"][i:i + 1], c["exps"][i:i + 1], 64)
        assert np.array_equal(yf, y - 2 * yi)


def test_plane_permutation(oracle_mod):
    c = workloads.random_case(4, 31, 256, 128, 2, seed=61, outlier_fraction=0.01)
    y, a = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128)
    perm = [2, 0, 3, 1]
    yp, ap = oracle_mod.shiftadd_gemm(c["x"], c["signs"][perm], c["exps"][perm], 128)
    assert np.all(np.abs(yp - y) <= 4 * 2.0 ** -52 * a)
    assert np.allclose(ap, a, rtol=1e-15, atol=0)


def test_special_case_pm1_matvec(oracle_mod):
    """q=1, e=0, G=K: the textbook +-1 matrix-vector product."""
    c = workloads.random_case(1, 50, 320, 320, 3, seed=71)
    e0 = np.zeros_like(c["exps"])
    y, a = oracle_mod.shiftadd_gemm(c["x"], c["signs"], e0, 320)
    x = c["x"].astype(np.float64)
    assert np.array_equal(y, x @ c["signs"][0].astype(np.float64).T)
    assert np.array_equal(a, np.repeat(np.abs(x).sum(1, keepdims=True), 50, axis=1))


def test_all_plus_ones(oracle_mod):
    c = workloads.random_case(3, 7, 256, 64, 2, seed=81)
    s = np.ones_like(c["signs"])
    y, a = oracle_mod.shiftadd_gemm(c["x"], s, c["exps"], 64)
    x = c["x"].astype(np.float64)
    gs = x.reshape(2, 4, 64).sum(-1)  # [B][NG]
    want = np.einsum("bg,ing->bn", gs, np.ldexp(1.0, c["exps"].astype(np.int64)))
    assert np.allclose(y, want, rtol=0, atol=1e-13 * a.max())


def test_rows_variant_matches_full(oracle_mod):
    c = workloads.random_case(2, 100, 256, 128, 3, seed=91)
    y, a = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128)
    rows = [0, 5, 99, 42, 42]
    yr, ar = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128, rows=rows)
    assert np.array_equal(yr, y[:, rows]) and np.array_equal(ar, a[:, rows])


def test_thread_count_does_not_change_results(oracle_mod):
    c = workloads.random_case(3, 64, 512, 128, 2, seed=92)
    y1, _ = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128, nthreads=1)
    y4, _ = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128, nthreads=4)
    assert np.array_equal(y1, y4)


# ----------------------------------------------------------------------------- mutants

def _definition(case, mutant=None):
    """The layer written out in numpy, with an optional planted mistake.

    Only used to show that the pins above reject plausible mistakes; the oracle
    itself is the C code.
    """
    s = case["signs"].astype(np.float64)
    e = case["exps"].astype(np.int64)
    G = case["G"]
    q, N, K = s.shape
    x = case["x"].astype(np.float64)
    if mutant == "drop_last_plane":
        s, e, q = s[:-1], e[:-1], q - 1
    if mutant == "flip_sign":
        s = -s
    if mutant == "negated_exponent":
        e = -e
    if mutant == "group_index_modulo":  # k % NG instead of k // G
        idx = np.arange(K) % (K // G)
    elif mutant == "group_off_by_one":
        idx = np.minimum((np.arange(K) + 1) // G, K // G - 1)
    else:
        idx = np.arange(K) // G
    scale = np.ldexp(1.0, e[:, :, idx])
    if mutant == "transposed_x":  # reversed column order inside each chunk
        x = x.reshape(x.shape[0], -1, 8)[:, :, ::-1].reshape(x.shape)
    y = np.einsum("bk,ink->bn", x, scale * s)
    if mutant == "dropped_term":  # last column of every row ignored
        y = y - np.einsum("b,in->bn", x[:, -1], (scale * s)[:, :, -1])
    return y


MUTANTS = ["drop_last_plane", "flip_sign", "negated_exponent", "group_index_modulo",
           "group_off_by_one", "transposed_x", "dropped_term"]


def test_definition_copy_agrees_with_pins(oracle_mod):
    c = workloads.random_case(3, 20, 256, 64, 2, seed=101, exp_range=(-6, 3))
    yd, ad = _dense(c)
    assert np.all(np.abs(_definition(c) - yd) <= 1e-12 * ad)


@pytest.mark.parametrize("mutant", MUTANTS)
def test_pins_reject_mutant(oracle_mod, mutant):
    c = workloads.random_case(3, 20, 256, 64, 2, seed=101, exp_range=(-6, 3))
    yd, ad = _dense(c)
    ym = _definition(c, mutant)
    assert not np.all(np.abs(ym - yd) <= 1e-12 * ad), mutant


def _lut_mutant(x, mutant):
    x = np.asarray(x, np.float64)
    B, K = x.shape
    bits = _bits256()
    if mutant == "msb_first":
        bits = bits[:, ::-1]
    sign = 2 * bits - 1
    if mutant == "bit_means_minus":
        sign = -sign
    xc = x.reshape(B, K // 8, 8)
    if mutant == "dropped_element":
        xc = xc.copy()
        xc[..., 7] = 0
    return np.einsum("mj,bcj->bcm", sign, xc)


@pytest.mark.parametrize("mutant", ["msb_first", "bit_means_minus", "dropped_element"])
def test_lut_pins_reject_mutant(mutant):
    h = _hand()["lut_chunk"]
    t = _lut_mutant(np.array([h["x"]], np.float16), mutant)[0, 0]
    assert any(t[int(k)] != v for k, v in h["entries"].items()), mutant
