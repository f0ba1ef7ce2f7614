"""The packed device layout declared in include/shiftadd.h, restated in numpy.

Used by tests to map device bytes to the canonical [q][N][K/8] key order.  The
CPU tests check this restatement against the library's sa_packed_offset.
"""
import numpy as np


def offsets(q: int, N: int, K: int) -> np.ndarray:
    """int64 [q][N][K/8]: byte offset of key (i, n, c) in the packed buffer."""
    C = K // 8
    i = np.arange(q, dtype=np.int64)[:, None, None]
    n = np.arange(N, dtype=np.int64)[None, :, None]
    c = np.arange(C, dtype=np.int64)[None, None, :]
    T, r = n // 64, n % 64
    R = np.minimum(64, N - 64 * T)
    J, u = c // 16, c % 16
    U = np.minimum(16, C - 16 * J)
    p = np.where(U == 16, (u - r) % 16, u)
    return (i * N + 64 * T) * C + 16 * J * R + r * U + p


def to_canonical(packed: np.ndarray, q: int, N: int, K: int) -> np.ndarray:
    return np.asarray(packed).reshape(-1)[offsets(q, N, K)]
