"""CPU oracle for the ShiftAddLLM shift-add linear layer (fp64).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(``paper_2406_05981_amd``) never imports it and shares no code with it.

The arithmetic lives in ``oracle.c`` (plain fp64 C, OpenMP over outputs); this
module only builds and loads it and marshals numpy arrays.  What each function
computes, with the passage it follows:

* :func:`pack` / :func:`unpack` -- the 8-bit keys of Sec. 4.1 (eight binary
  weights of a plane row index one table): byte c of a plane row is
  ``sum_j [s[8c+j] > 0] << j``; bit value 1 stands for +1 (a reading: the paper
  does not fix the bit order or the bit-to-sign map).
* :func:`lut` -- the 256 precomputed partial sums per 8 activations of Sec. 4.1:
  ``lut[b][c][m] = sum_j (2 bit_j(m) - 1) x[b][8c+j]``.
* :func:`shiftadd_gemm` -- the layer ``y = x W_q^T`` with
  ``W_q = sum_i 2^{e_i} b_i`` (Sec. 3 BCQ with the power-of-two factors of
  Eq. 2, one factor per plane, row and group of G columns), and the sum of the
  magnitudes of its terms (the tolerance reference).
* :func:`shiftadd_gemm_colwise` -- the layer with column-wise scaling factors
  ("Ours (Acc.)", Sec. 4.2): one power-of-two factor per plane and weight
  column, ``W_q[n][k] = sum_i 2^{e_i[k]} b_i[n][k]``, so that
  ``y = sum_i sum_k b_i[n][k] 2^{e_i[k]} x[k]`` (the factor shifts the
  activation it meets).
* :func:`shiftadd_gemm_blockwise` -- the layer with block-wise scaling factors
  ("Ours (Lat.)", Sec. 4.2): 8 columns (one key) and a block of ``row_block``
  rows share one power-of-two factor,
  ``y = sum_i sum_c ldexp(sum_{j<8} b_i[n][8c+j] x[8c+j], E[i][n // row_block][c])``.
* :func:`shiftadd_gemm_terms` -- the layer with additive power-of-two factors
  (Eq. 2 with T terms): the factor of (plane, row, group) is
  ``sum_t sg_t 2^{e_t}``, term signs in {-1, 0, +1} (0: no term).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` with gcc into ``liboracle.so`` next to it."""
    if not force and os.path.exists(_LIB_PATH) and \
            os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC):
        return _LIB_PATH
    tmp = _LIB_PATH + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wextra",
           "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def build_sanitized(out: str) -> str:
    """Compile ``oracle.c`` with AddressSanitizer and UndefinedBehaviorSanitizer
    (gcc) into ``out``; a process loading it must preload gcc's libasan.  Set
    ``ORACLE_LIB`` to its path to make this module load it."""
    tmp = out + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp", "-fPIC", "-shared",
           "-std=c11", "-Wall", "-Wextra", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = os.environ.get("ORACLE_LIB")   # another build of oracle.c (the sanitized one)
    if not path:
        build(force=False)
        path = _LIB_PATH
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    lib.oracle_max_threads.argtypes = [ctypes.c_int]
    lib.oracle_max_threads.restype = ctypes.c_int
    lib.oracle_pack.argtypes = [P, I64, I64, I64, P]
    lib.oracle_pack.restype = None
    lib.oracle_unpack.argtypes = [P, I64, I64, I64, P]
    lib.oracle_unpack.restype = None
    lib.oracle_lut.argtypes = [P, I64, I64, P]
    lib.oracle_lut.restype = None
    lib.oracle_shiftadd_gemm.argtypes = [P, P, P, I64, I64, I64, I64, I64, P, P, ctypes.c_int]
    lib.oracle_shiftadd_gemm.restype = None
    lib.oracle_shiftadd_gemm_rows.argtypes = [P, P, P, I64, I64, I64, I64, I64, P, I64,
                                              P, P, ctypes.c_int]
    lib.oracle_shiftadd_gemm_rows.restype = None
    lib.oracle_shiftadd_gemm_colwise.argtypes = [P, P, P, I64, I64, I64, I64, P, I64,
                                                 P, P, ctypes.c_int]
    lib.oracle_shiftadd_gemm_colwise.restype = None
    lib.oracle_shiftadd_gemm_blockwise.argtypes = [P, P, P, I64, I64, I64, I64, I64, P, I64,
                                                   P, P, ctypes.c_int]
    lib.oracle_shiftadd_gemm_blockwise.restype = None
    lib.oracle_shiftadd_gemm_terms.argtypes = [P, P, P, P, I64, I64, I64, I64, I64, I64, P,
                                               I64, P, P, ctypes.c_int]
    lib.oracle_shiftadd_gemm_terms.restype = None
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def _check_shapes(signs: np.ndarray, exps: np.ndarray, x: np.ndarray, G: int):
    q, N, K = signs.shape
    B = x.shape[0]
    if K % 8 or G % 8 or K % G:
        raise ValueError(f"need K % 8 == 0, G % 8 == 0, K % G == 0 (K={K}, G={G})")
    if exps.shape != (q, N, K // G):
        raise ValueError(f"exps shape {exps.shape} != {(q, N, K // G)}")
    if x.shape != (B, K):
        raise ValueError(f"x shape {x.shape} != {(B, K)}")
    return q, N, K, B


def max_threads(nthreads: int = 0) -> int:
    return int(_load().oracle_max_threads(int(nthreads)))


def pack(signs: np.ndarray) -> np.ndarray:
    """Canonical packed planes ``uint8 [q][N][K/8]`` of ``int8 [q][N][K]`` signs."""
    signs = np.ascontiguousarray(signs, dtype=np.int8)
    q, N, K = signs.shape
    if K % 8:
        raise ValueError("K must be a multiple of 8")
    out = np.empty((q, N, K // 8), dtype=np.uint8)
    _load().oracle_pack(_ptr(signs), q, N, K, _ptr(out))
    return out


def unpack(packed: np.ndarray, K: int) -> np.ndarray:
    """Inverse of :func:`pack`: ``int8 [q][N][K]`` in {-1, +1}."""
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    q, N, C = packed.shape
    if C * 8 != K:
        raise ValueError("packed.shape[2] * 8 must equal K")
    out = np.empty((q, N, K), dtype=np.int8)
    _load().oracle_unpack(_ptr(packed), q, N, K, _ptr(out))
    return out


def lut(x: np.ndarray) -> np.ndarray:
    """Tables ``fp64 [B][K/8][256]`` of the activations ``x [B][K]`` (fp16 or wider)."""
    x64 = np.ascontiguousarray(np.asarray(x).astype(np.float64))
    B, K = x64.shape
    if K % 8:
        raise ValueError("K must be a multiple of 8")
    out = np.empty((B, K // 8, 256), dtype=np.float64)
    _load().oracle_lut(_ptr(x64), B, K, _ptr(out))
    return out


def shiftadd_gemm(x: np.ndarray, signs: np.ndarray, exps: np.ndarray, G: int,
                  nthreads: int = 0, rows: Optional[Sequence[int]] = None
                  ) -> Tuple[np.ndarray, np.ndarray]:
    """``(y, absterm)``, both fp64 ``[B][N]`` (or ``[B][len(rows)]``).

    ``y[b][n] = sum_i sum_g ldexp(sum_{k in g} s_i[n][k] x[b][k], e[i][n][g])`` and
    ``absterm[b][n] = sum_i sum_k 2^e |x[b][k]|``.
    """
    x64 = np.ascontiguousarray(np.asarray(x).astype(np.float64))
    signs = np.ascontiguousarray(signs, dtype=np.int8)
    exps = np.ascontiguousarray(exps, dtype=np.int8)
    q, N, K, B = _check_shapes(signs, exps, x64, G)
    lib = _load()
    if rows is None:
        y = np.empty((B, N), dtype=np.float64)
        a = np.empty((B, N), dtype=np.float64)
        lib.oracle_shiftadd_gemm(_ptr(x64), _ptr(signs), _ptr(exps), q, N, K, G, B,
                                 _ptr(y), _ptr(a), int(nthreads))
    else:
        r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        if r.size and (r.min() < 0 or r.max() >= N):
            raise ValueError("row index out of range")
        y = np.empty((B, r.size), dtype=np.float64)
        a = np.empty((B, r.size), dtype=np.float64)
        lib.oracle_shiftadd_gemm_rows(_ptr(x64), _ptr(signs), _ptr(exps), q, N, K, G, B,
                                      _ptr(r), r.size, _ptr(y), _ptr(a), int(nthreads))
    return y, a


def shiftadd_gemm_colwise(x: np.ndarray, signs: np.ndarray, col_exps: np.ndarray,
                          nthreads: int = 0, rows: Optional[Sequence[int]] = None
                          ) -> Tuple[np.ndarray, np.ndarray]:
    """``(y, absterm)``, fp64 ``[B][N]`` (or ``[B][len(rows)]``), of the layer with
    column-wise factors: ``y[b][n] = sum_i sum_k s_i[n][k] ldexp(x[b][k], e[i][k])``
    and ``absterm[b][n] = sum_i sum_k 2^e[i][k] |x[b][k]|``."""
    x64 = np.ascontiguousarray(np.asarray(x).astype(np.float64))
    signs = np.ascontiguousarray(signs, dtype=np.int8)
    col_exps = np.ascontiguousarray(col_exps, dtype=np.int8)
    q, N, K = signs.shape
    B = x64.shape[0]
    if col_exps.shape != (q, K):
        raise ValueError(f"col_exps shape {col_exps.shape} != {(q, K)}")
    if x64.shape != (B, K):
        raise ValueError(f"x shape {x64.shape} != {(B, K)}")
    lib = _load()
    if rows is None:
        r, R, rp = None, N, None
    else:
        r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        if r.size and (r.min() < 0 or r.max() >= N):
            raise ValueError("row index out of range")
        R, rp = r.size, _ptr(r)
    y = np.empty((B, R), dtype=np.float64)
    a = np.empty((B, R), dtype=np.float64)
    lib.oracle_shiftadd_gemm_colwise(_ptr(x64), _ptr(signs), _ptr(col_exps), q, N, K, B,
                                     rp, R if r is not None else 0, _ptr(y), _ptr(a),
                                     int(nthreads))
    return y, a


def shiftadd_gemm_blockwise(x: np.ndarray, signs: np.ndarray, blk_exps: np.ndarray,
                            row_block: int, nthreads: int = 0,
                            rows: Optional[Sequence[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """``(y, absterm)``, fp64 ``[B][N]`` (or ``[B][len(rows)]``), of the layer with
    block-wise factors ``E int8 [q][ceil(N / row_block)][K / 8]``:
    ``y[b][n] = sum_i sum_c ldexp(sum_j s_i[n][8c+j] x[b][8c+j], E[i][n // row_block][c])``."""
    x64 = np.ascontiguousarray(np.asarray(x).astype(np.float64))
    signs = np.ascontiguousarray(signs, dtype=np.int8)
    blk_exps = np.ascontiguousarray(blk_exps, dtype=np.int8)
    q, N, K = signs.shape
    B = x64.shape[0]
    NB = -(-N // row_block)
    if K % 8 or blk_exps.shape != (q, NB, K // 8):
        raise ValueError(f"blk_exps shape {blk_exps.shape} != {(q, NB, K // 8)}")
    if x64.shape != (B, K):
        raise ValueError(f"x shape {x64.shape} != {(B, K)}")
    lib = _load()
    if rows is None:
        r, R, rp = None, N, None
    else:
        r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        if r.size and (r.min() < 0 or r.max() >= N):
            raise ValueError("row index out of range")
        R, rp = r.size, _ptr(r)
    y = np.empty((B, R), dtype=np.float64)
    a = np.empty((B, R), dtype=np.float64)
    lib.oracle_shiftadd_gemm_blockwise(_ptr(x64), _ptr(signs), _ptr(blk_exps), q, N, K,
                                       row_block, B, rp, R if r is not None else 0, _ptr(y),
                                       _ptr(a), int(nthreads))
    return y, a


def shiftadd_gemm_terms(x: np.ndarray, signs: np.ndarray, exps: np.ndarray,
                        term_signs: np.ndarray, G: int, nthreads: int = 0,
                        rows: Optional[Sequence[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """``(y, absterm)`` of the layer with additive power-of-two factors:
    ``exps, term_signs int8 [q][N][K/G][T]``,
    ``y[b][n] = sum_i sum_g sum_t sg_t ldexp(sum_{k in g} s_i[n][k] x[b][k], e_t)``."""
    x64 = np.ascontiguousarray(np.asarray(x).astype(np.float64))
    signs = np.ascontiguousarray(signs, dtype=np.int8)
    exps = np.ascontiguousarray(exps, dtype=np.int8)
    term_signs = np.ascontiguousarray(term_signs, dtype=np.int8)
    q, N, K = signs.shape
    B = x64.shape[0]
    T = exps.shape[-1]
    if K % 8 or G % 8 or K % G or exps.shape != (q, N, K // G, T) or term_signs.shape != exps.shape:
        raise ValueError(f"exps/term_signs shape {exps.shape}/{term_signs.shape} != "
                         f"{(q, N, K // G, T)}")
    if x64.shape != (B, K):
        raise ValueError(f"x shape {x64.shape} != {(B, K)}")
    lib = _load()
    if rows is None:
        r, R, rp = None, N, None
    else:
        r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        if r.size and (r.min() < 0 or r.max() >= N):
            raise ValueError("row index out of range")
        R, rp = r.size, _ptr(r)
    y = np.empty((B, R), dtype=np.float64)
    a = np.empty((B, R), dtype=np.float64)
    lib.oracle_shiftadd_gemm_terms(_ptr(x64), _ptr(signs), _ptr(exps), _ptr(term_signs), T, q,
                                   N, K, G, B, rp, R if r is not None else 0, _ptr(y), _ptr(a),
                                   int(nthreads))
    return y, a
