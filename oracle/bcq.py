"""CPU oracle for the offline reparameterization of ShiftAddLLM (fp64, numpy).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  The product path
(``paper_2406_05981_amd``) never imports it and shares no code with it.

What it computes (parity is pinned by ``tests/test_bcq_oracle.py``): a weight
matrix W [N][K] is cut into segments of G consecutive columns of one row (the
groups of the shift-add layer, one power-of-two factor per plane, row and
group), and every segment w in R^G is quantized by the alternating multi-bit
binary-coding quantization of Sec. 3 (Alg. 1) with the power-of-two scale
factors of Sec. 4.1 (Eq. 2, one term):

* ``greedy`` -- Eq. 1: r_0 = w; for i = 1..q: b_i = sign(r_{i-1}),
  alpha_i = r_{i-1}^T b_i / G, r_i = r_{i-1} - alpha_i b_i.
* ``least_squares`` -- the LS step: alpha = (B^T B)^{-1} B^T w with
  B = [b_1 .. b_q].
* ``pot`` -- Eq. 2 with one term: alpha -> sign(alpha) 2^P,
  P = round(log2 |alpha|).
* ``binary_search`` -- the BS step: with alpha fixed, each element takes the
  codes whose value sum_i alpha_i b_i is nearest to it (the binary search over
  the sorted 2^q representable values finds exactly this nearest value).
* ``pot_terms`` -- Eq. 2 with several terms (additive PoT): term t is the PoT
  of the residual alpha - sum_{j<t} a_j.
* ``quantize`` -- greedy initialisation, then T cycles of LS, PoT, BS; the
  output is the hot-path format: planes s_i = sign(alpha_i) b_i (the sign of the
  factor folded into the plane) and int8 exponents e_i = P_i, so that
  W_q = sum_i 2^{e_i} s_i per segment.

Readings where the paper is silent:

* sign(0) = +1.
* PoT is applied to the scales that BS uses (after every LS step) and to the
  greedy scales when T = 0, because the output format holds powers of two only.
* round(log2 |a|): with |a| = m 2^E, m in [1, 2), P = E + [m >= sqrt(2)]
  (log-domain rounding; m = sqrt(2) cannot occur in floating point, so there
  are no ties); a = 0 gives P = -128 and sign +1; P is clamped to [-128, 127].
* LS when B^T B is singular: Gaussian elimination with partial pivoting over
  the columns in order; a column whose best pivot is at most 1e-9 * G in
  magnitude depends on the earlier ones and gets alpha = 0.  The rest is the
  exact least-squares solution of the remaining columns.
* BS ties (two code vectors at the same distance): the one with the smaller
  code number, where code c has b_i = +1 exactly when bit i of c is set.

Everything is vectorised over segments only; each step is the definition above
written out, in the order the paper gives.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

SQRT2 = np.sqrt(2.0)
P_MIN, P_MAX = -128, 127


def segments(w: np.ndarray, group: int) -> np.ndarray:
    """[N][K] -> [N * K/group][group] fp64, row-major over (row, group)."""
    N, K = w.shape
    return np.asarray(w, np.float64).reshape(N * (K // group), group)


def sign_pm1(r: np.ndarray) -> np.ndarray:
    return np.where(r >= 0, 1.0, -1.0)


def greedy(w: np.ndarray, q: int) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. 1 on every segment: codes [S][q][G] (+-1) and scales [S][q]."""
    S, G = w.shape
    r = w.copy()
    B = np.empty((S, q, G))
    A = np.empty((S, q))
    for i in range(q):
        B[:, i] = sign_pm1(r)
        A[:, i] = (r * B[:, i]).sum(axis=1) / G
        r = r - A[:, i:i + 1] * B[:, i]
    return B, A


def least_squares(B: np.ndarray, w: np.ndarray) -> np.ndarray:
    """alpha = (B^T B)^{-1} B^T w on every segment (reading for singular B^T B
    in the module docstring), by Gaussian elimination with partial pivoting."""
    S, q, G = B.shape
    M = np.einsum("sig,sjg->sij", B, B)            # integers, exact
    v = np.einsum("sig,sg->si", B, w)
    tol = 1e-9 * G
    alpha = np.zeros((S, q))
    for s in range(S):
        a = M[s].copy()
        rhs = v[s].copy()
        pivot_row = []                              # (row, column) per kept column
        row = 0
        for col in range(q):
            if row == q:
                break
            p = row + int(np.argmax(np.abs(a[row:, col])))
            if abs(a[p, col]) <= tol:
                continue                            # dependent column: alpha = 0
            if p != row:
                a[[row, p]] = a[[p, row]]
                rhs[[row, p]] = rhs[[p, row]]
            for r2 in range(row + 1, q):
                f = a[r2, col] / a[row, col]
                a[r2] = a[r2] - f * a[row]
                rhs[r2] = rhs[r2] - f * rhs[row]
            pivot_row.append((row, col))
            row += 1
        for row, col in reversed(pivot_row):
            acc = rhs[row]
            for r2, c2 in pivot_row:
                if c2 > col:
                    acc = acc - a[row, c2] * alpha[s, c2]
            alpha[s, col] = acc / a[row, col]
    return alpha


def pot(alpha: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. 2 with one term: (sign, P) with alpha ~ sign * 2^P."""
    mag = np.abs(alpha)
    m, E = np.frexp(mag)                            # mag = m 2^E, m in [0.5, 1)
    P = (E - 1) + (2.0 * m >= SQRT2)
    P = np.where(mag == 0, P_MIN, np.clip(P, P_MIN, P_MAX)).astype(np.int64)
    sgn = np.where(alpha < 0, -1.0, 1.0)
    return sgn, P


def pot_values(alpha: np.ndarray) -> np.ndarray:
    sgn, P = pot(alpha)
    return np.where(np.abs(alpha) == 0, 0.0, sgn * np.ldexp(1.0, P))


def pot_terms(alpha: np.ndarray, terms: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Additive PoT (Eq. 2 with ``terms`` terms): term t rounds the residual
    of the previous terms, a_t = POT(alpha - sum_{j<t} a_j).  Returns the
    value sum_t a_t (summed in term order from 0), and the per-term signs
    (+-1, 0 for a zero residual) and exponents P_t, each [terms][...]."""
    r = np.asarray(alpha, np.float64).copy()
    val = np.zeros_like(r)
    sgns = np.empty((terms,) + r.shape)
    Ps = np.empty((terms,) + r.shape, dtype=np.int64)
    for t in range(terms):
        sg, P = pot(r)
        a_t = pot_values(r)
        sgns[t] = np.where(r == 0, 0.0, sg)
        Ps[t] = P
        val = val + a_t
        r = r - a_t
    return val, sgns, Ps


def code_values(a: np.ndarray) -> np.ndarray:
    """value[s][c] = sum_i a[s][i] (bit i of c ? +1 : -1), summed in plane order."""
    S, q = a.shape
    vals = np.zeros((S, 1 << q))
    for c in range(1 << q):
        acc = np.zeros(S)
        for i in range(q):
            acc = acc + (a[:, i] if (c >> i) & 1 else -a[:, i])
        vals[:, c] = acc
    return vals


def binary_search(a: np.ndarray, w: np.ndarray) -> np.ndarray:
    """The BS step: nearest representable value per element; codes [S][q][G]."""
    S, q = a.shape
    vals = code_values(a)                          # [S][2^q]
    dist = np.abs(w[:, :, None] - vals[:, None, :])  # [S][G][2^q]
    best = np.argmin(dist, axis=2)                 # first minimum = smallest code
    B = np.empty((S, q, w.shape[1]))
    for i in range(q):
        B[:, i] = np.where((best >> i) & 1, 1.0, -1.0)
    return B


def quantize_segments(w: np.ndarray, q: int, cycles: int, trace: bool = False, terms: int = 1):
    """Alg. 1 with PoT scales (``terms`` additive terms each) on segments
    [S][G]; returns (B, PoT alphas) -- and the per-error trace when asked."""
    B, A, pa, errors = _alternate(w, q, cycles, terms, trace)
    return (B, pa, errors) if trace else (B, pa)


def _alternate(w: np.ndarray, q: int, cycles: int, terms: int, trace: bool = False):
    """The steps of Alg. 1: (codes B, the last unrounded scales A, their PoT
    values pa, error trace)."""
    B, A = greedy(w, q)
    errors = []
    if trace:
        errors.append(np.square(w - np.einsum("si,sig->sg", A, B)).sum(axis=1))
    rounded = (lambda a: pot_values(a)) if terms == 1 else (lambda a: pot_terms(a, terms)[0])
    pa = rounded(A)
    for _ in range(cycles):
        A = least_squares(B, w)
        pa = rounded(A)
        B = binary_search(pa, w)
        if trace:
            errors.append(np.square(w - np.einsum("si,sig->sg", pa, B)).sum(axis=1))
    return B, A, pa, errors


def quantize(w: np.ndarray, q: int, group: int, cycles: int):
    """W [N][K] -> (signs int8 [q][N][K], exps int8 [q][N][K/group]) in the
    layer's format: W_q[n][k] = sum_i 2^exps[i][n][k/group] * signs[i][n][k]."""
    N, K = w.shape
    NG = K // group
    B, pa = quantize_segments(segments(w, group), q, cycles)
    sgn, P = pot(pa)
    signs = (B * sgn[:, :, None]).astype(np.int8)   # [S][q][G]
    signs = signs.reshape(N, NG, q, group).transpose(2, 0, 1, 3).reshape(q, N, K)
    exps = P.astype(np.int8).reshape(N, NG, q).transpose(2, 0, 1)
    return np.ascontiguousarray(signs), np.ascontiguousarray(exps)


def quantize_terms(w: np.ndarray, q: int, group: int, cycles: int, terms: int):
    """W [N][K] -> (signs int8 [q][N][K], exps int8 [q][N][K/group][terms],
    term_signs int8 [q][N][K/group][terms]) with additive PoT scales: the
    scale of (plane, row, group) is sum_t term_signs[..., t] 2^exps[..., t].  The sign of
    the first term is folded into the plane (a zero scale keeps the plane's
    codes and gets term sign 0), so term 0 has sign +1 or 0 and later terms
    carry their sign relative to it."""
    N, K = w.shape
    NG = K // group
    B, A, pa, _ = _alternate(segments(w, group), q, cycles, terms)
    _, sg, P = pot_terms(A, terms)                     # [T][S][q]
    s0 = np.where(sg[0] < 0, -1.0, 1.0)               # [S][q]
    signs = (B * s0[:, :, None]).astype(np.int8)
    signs = signs.reshape(N, NG, q, group).transpose(2, 0, 1, 3).reshape(q, N, K)
    tsg = (sg * s0[None]).astype(np.int8)             # term 0 -> +1 (or 0)
    exps = P.astype(np.int8).reshape(terms, N, NG, q).transpose(3, 1, 2, 0)
    tsg = tsg.reshape(terms, N, NG, q).transpose(3, 1, 2, 0)
    return np.ascontiguousarray(signs), np.ascontiguousarray(exps), np.ascontiguousarray(tsg)


def reconstruct_terms(signs: np.ndarray, exps: np.ndarray, term_signs: np.ndarray,
                      group: int) -> np.ndarray:
    """W_q [N][K] = sum_i (sum_t term_signs[..., t] 2^exps[..., t]) * signs, in fp64."""
    f = (term_signs.astype(np.float64) * np.ldexp(1.0, exps.astype(np.int64))).sum(axis=-1)
    return (np.repeat(f, group, axis=2) * signs).sum(axis=0)


def reconstruct(signs: np.ndarray, exps: np.ndarray, group: int) -> np.ndarray:
    """W_q [N][K] = sum_i 2^exps * signs, in fp64."""
    q, N, K = signs.shape
    scale = np.ldexp(1.0, np.repeat(exps.astype(np.int64), group, axis=2))
    return (scale * signs).sum(axis=0)
