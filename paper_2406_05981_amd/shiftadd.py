"""Python binding of ``libshiftadd.so`` (argument marshalling only).

Every function has the name of the C entry point it calls (see
``include/shiftadd.h``).  Tensors must live on the current HIP device; torch is
used for device memory and streams only -- every step of the layer runs in the
library's HIP kernels.  A missing library raises at import; a rejected call
raises :class:`SaError` with the library's status text.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# SHIFTADD_LIB selects another build of the same sources (the sanitized host
# build of the CPU tests); by default the in-tree library
LIB_PATH = os.environ.get("SHIFTADD_LIB") or os.path.join(_HERE, "libshiftadd.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with `python -m paper_2406_05981_amd.build` "
        "(there is no fallback path)")


class SaPlan(ctypes.Structure):
    _fields_ = [
        ("path", ctypes.c_int),
        ("rows_per_wg", ctypes.c_int),
        ("workgroups", ctypes.c_int),
        ("threads", ctypes.c_int),
        ("pieces", ctypes.c_int),
        ("lds_bytes", ctypes.c_size_t),
    ]


def _bind(lib):
    P = ctypes.c_void_p
    I = ctypes.c_int
    sig = {
        "sa_packed_bytes": ([I, I, I], ctypes.c_size_t),
        "sa_packed_offset": ([I, I, I, I, I, I], ctypes.c_int64),
        "sa_pack_weights": ([P, I, I, I, P, P], I),
        "sa_unpack_weights": ([P, I, I, I, P, P], I),
        "sa_build_lut": ([P, I, I, P, P], I),
        "sa_shiftadd_gemm": ([P, P, P, I, I, I, I, I, P, P], I),
        "sa_shiftadd_gemm_f16": ([P, P, P, I, I, I, I, I, P, P], I),
        "sa_plan_gemm": ([I, I, I, I, I, ctypes.POINTER(SaPlan)], I),
        "sa_kslice_workspace_bytes": ([I, I], ctypes.c_size_t),
        "sa_shiftadd_gemm_kslice": ([P, P, P, I, I, I, I, P, P, ctypes.c_size_t, P], I),
        "sa_shiftadd_gemm_colwise": ([P, P, P, I, I, I, I, P, P], I),
        "sa_plan_gemm_colwise": ([I, I, I, I, ctypes.POINTER(SaPlan)], I),
        "sa_shiftadd_gemm_blockwise": ([P, P, P, I, I, I, I, I, P, P], I),
        "sa_plan_gemm_blockwise": ([I, I, I, I, I, ctypes.POINTER(SaPlan)], I),
        "sa_shiftadd_gemm_terms": ([P, P, P, P, I, I, I, I, I, I, P, P], I),
        "sa_read_probe": ([P, ctypes.c_size_t, P, P], I),
        "sa_quantize_bcq": ([P, I, I, I, I, I, P, P, P], I),
        "sa_quantize_bcq_terms": ([P, I, I, I, I, I, I, P, P, P, P], I),
        "sa_gram_f16": ([P, I, I, P, P], I),
        "sa_inverse_cholesky_workspace": ([I], ctypes.c_size_t),
        "sa_inverse_cholesky_diag": ([P, I, ctypes.c_double, P, P, ctypes.c_size_t, P], I),
        "sa_importance_workspace": ([], ctypes.c_size_t),
        "sa_importance_criterion": ([P, I, I, P, P, P, ctypes.c_size_t, P], I),
        "sa_importance_criterion_noalloc": ([P, I, I, P, P, P], I),
        "sa_fit_per_bit": ([P, P, I, I, I, P], I),
        "sa_allocate_bits": ([P, P, I, I, ctypes.c_double, P, P], I),
        "sa_status_string": ([I], ctypes.c_char_p),
        "sa_version": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    return lib


lib = _bind(ctypes.CDLL(LIB_PATH))

SA_OK, SA_ERR_NULL, SA_ERR_SHAPE, SA_ERR_Q, SA_ERR_GROUP, SA_ERR_ALIGN, SA_ERR_HIP = (
    0, -1, -2, -3, -4, -5, -6)
SA_MAX_Q = 8
SA_MAX_BATCH = 256
SA_MAX_CYCLES = 64
SA_MAX_TERMS = 4


class SaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {sa_status_string(status)} (status {status})")


def _check(status: int, where: str) -> None:
    if status != SA_OK:
        raise SaError(status, where)


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _dev(t: torch.Tensor, name: str, dtype: torch.dtype, numel: int) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() != numel:
        raise ValueError(f"{name} must have {numel} elements, got {t.numel()}")
    return t.data_ptr()


def sa_status_string(status: int) -> str:
    return lib.sa_status_string(int(status)).decode()


def sa_version() -> str:
    return lib.sa_version().decode()


def sa_packed_bytes(q: int, N: int, K: int) -> int:
    return int(lib.sa_packed_bytes(q, N, K))


def sa_packed_offset(q: int, N: int, K: int, i: int, n: int, c: int) -> int:
    return int(lib.sa_packed_offset(q, N, K, i, n, c))


def sa_plan_gemm(q: int, N: int, K: int, group: int, batch: int) -> dict:
    p = SaPlan()
    _check(lib.sa_plan_gemm(q, N, K, group, batch, ctypes.byref(p)), "sa_plan_gemm")
    return {name: getattr(p, name) for name, _ in SaPlan._fields_}


def sa_plan_gemm_colwise(q: int, N: int, K: int, batch: int) -> dict:
    p = SaPlan()
    _check(lib.sa_plan_gemm_colwise(q, N, K, batch, ctypes.byref(p)), "sa_plan_gemm_colwise")
    return {name: getattr(p, name) for name, _ in SaPlan._fields_}


def sa_plan_gemm_blockwise(q: int, N: int, K: int, row_block: int, batch: int) -> dict:
    p = SaPlan()
    _check(lib.sa_plan_gemm_blockwise(q, N, K, row_block, batch, ctypes.byref(p)),
           "sa_plan_gemm_blockwise")
    return {name: getattr(p, name) for name, _ in SaPlan._fields_}


def sa_pack_weights(signs: torch.Tensor, q: int, N: int, K: int, packed_bits: torch.Tensor,
                    stream=None) -> None:
    nbytes = sa_packed_bytes(q, N, K)
    if nbytes == 0:
        _check(SA_ERR_SHAPE if 1 <= q <= SA_MAX_Q else SA_ERR_Q, "sa_pack_weights")
    _check(lib.sa_pack_weights(_dev(signs, "signs", torch.int8, q * N * K), q, N, K,
                               _dev(packed_bits, "packed_bits", torch.uint8, nbytes),
                               _stream(stream)), "sa_pack_weights")


def sa_unpack_weights(packed_bits: torch.Tensor, q: int, N: int, K: int, signs: torch.Tensor,
                      stream=None) -> None:
    nbytes = sa_packed_bytes(q, N, K)
    if nbytes == 0:
        _check(SA_ERR_SHAPE if 1 <= q <= SA_MAX_Q else SA_ERR_Q, "sa_unpack_weights")
    _check(lib.sa_unpack_weights(_dev(packed_bits, "packed_bits", torch.uint8, nbytes), q, N, K,
                                 _dev(signs, "signs", torch.int8, q * N * K), _stream(stream)),
           "sa_unpack_weights")


def sa_build_lut(x: torch.Tensor, K: int, batch: int, lut: torch.Tensor, stream=None) -> None:
    _check(lib.sa_build_lut(_dev(x, "x", torch.float16, batch * K), K, batch,
                            _dev(lut, "lut", torch.float32, batch * (K // 8) * 256),
                            _stream(stream)), "sa_build_lut")


def sa_shiftadd_gemm(x: torch.Tensor, packed_bits: torch.Tensor, exps: torch.Tensor, q: int,
                     N: int, K: int, group: int, batch: int, y: torch.Tensor,
                     stream=None) -> None:
    if group <= 0 or K % group:
        _check(SA_ERR_GROUP, "sa_shiftadd_gemm")
    _check(lib.sa_shiftadd_gemm(
        _dev(x, "x", torch.float16, batch * K),
        _dev(packed_bits, "packed_bits", torch.uint8, sa_packed_bytes(q, N, K)),
        _dev(exps, "exps", torch.int8, q * N * (K // group)),
        q, N, K, group, batch,
        _dev(y, "y", torch.float32, batch * N), _stream(stream)), "sa_shiftadd_gemm")


def sa_shiftadd_gemm_f16(x: torch.Tensor, packed_bits: torch.Tensor, exps: torch.Tensor, q: int,
                         N: int, K: int, group: int, batch: int, y: torch.Tensor,
                         stream=None) -> None:
    if group <= 0 or K % group:
        _check(SA_ERR_GROUP, "sa_shiftadd_gemm_f16")
    _check(lib.sa_shiftadd_gemm_f16(
        _dev(x, "x", torch.float16, batch * K),
        _dev(packed_bits, "packed_bits", torch.uint8, sa_packed_bytes(q, N, K)),
        _dev(exps, "exps", torch.int8, q * N * (K // group)),
        q, N, K, group, batch,
        _dev(y, "y", torch.float16, batch * N), _stream(stream)), "sa_shiftadd_gemm_f16")


def sa_kslice_workspace_bytes(N: int, K: int) -> int:
    return int(lib.sa_kslice_workspace_bytes(N, K))


def sa_shiftadd_gemm_kslice(x: torch.Tensor, packed_bits: torch.Tensor, exps: torch.Tensor,
                            q: int, N: int, K: int, group: int, y: torch.Tensor,
                            workspace: torch.Tensor, stream=None) -> None:
    if group <= 0 or K % group:
        _check(SA_ERR_GROUP, "sa_shiftadd_gemm_kslice")
    _check(lib.sa_shiftadd_gemm_kslice(
        _dev(x, "x", torch.float16, K),
        _dev(packed_bits, "packed_bits", torch.uint8, sa_packed_bytes(q, N, K)),
        _dev(exps, "exps", torch.int8, q * N * (K // group)),
        q, N, K, group,
        _dev(y, "y", torch.float32, N),
        _dev(workspace, "workspace", torch.float32, workspace.numel()),
        4 * workspace.numel(), _stream(stream)), "sa_shiftadd_gemm_kslice")


def sa_shiftadd_gemm_colwise(x: torch.Tensor, packed_bits: torch.Tensor, col_exps: torch.Tensor,
                             q: int, N: int, K: int, batch: int, y: torch.Tensor,
                             stream=None) -> None:
    if sa_packed_bytes(q, N, K) == 0:
        _check(SA_ERR_SHAPE if 1 <= q <= SA_MAX_Q else SA_ERR_Q, "sa_shiftadd_gemm_colwise")
    _check(lib.sa_shiftadd_gemm_colwise(
        _dev(x, "x", torch.float16, batch * K),
        _dev(packed_bits, "packed_bits", torch.uint8, sa_packed_bytes(q, N, K)),
        _dev(col_exps, "col_exps", torch.int8, q * K),
        q, N, K, batch,
        _dev(y, "y", torch.float32, batch * N), _stream(stream)), "sa_shiftadd_gemm_colwise")


def sa_shiftadd_gemm_blockwise(x: torch.Tensor, packed_bits: torch.Tensor, blk_exps: torch.Tensor,
                               q: int, N: int, K: int, row_block: int, batch: int,
                               y: torch.Tensor, stream=None) -> None:
    if sa_packed_bytes(q, N, K) == 0:
        _check(SA_ERR_SHAPE if 1 <= q <= SA_MAX_Q else SA_ERR_Q, "sa_shiftadd_gemm_blockwise")
    if row_block < 1:
        _check(SA_ERR_SHAPE, "sa_shiftadd_gemm_blockwise")
    nb = -(-N // row_block)
    _check(lib.sa_shiftadd_gemm_blockwise(
        _dev(x, "x", torch.float16, batch * K),
        _dev(packed_bits, "packed_bits", torch.uint8, sa_packed_bytes(q, N, K)),
        _dev(blk_exps, "blk_exps", torch.int8, q * nb * (K // 8)),
        q, N, K, row_block, batch,
        _dev(y, "y", torch.float32, batch * N), _stream(stream)), "sa_shiftadd_gemm_blockwise")


def sa_shiftadd_gemm_terms(x: torch.Tensor, packed_bits: torch.Tensor, exps: torch.Tensor,
                           term_signs: torch.Tensor, q: int, N: int, K: int, group: int,
                           terms: int, batch: int, y: torch.Tensor, stream=None) -> None:
    if sa_packed_bytes(q, N, K) == 0:
        _check(SA_ERR_SHAPE if 1 <= q <= SA_MAX_Q else SA_ERR_Q, "sa_shiftadd_gemm_terms")
    if group <= 0 or K % group:
        _check(SA_ERR_GROUP, "sa_shiftadd_gemm_terms")
    if terms < 1 or terms > SA_MAX_TERMS:
        _check(SA_ERR_SHAPE, "sa_shiftadd_gemm_terms")
    n_e = terms * q * N * (K // group)
    _check(lib.sa_shiftadd_gemm_terms(
        _dev(x, "x", torch.float16, batch * K),
        _dev(packed_bits, "packed_bits", torch.uint8, sa_packed_bytes(q, N, K)),
        _dev(exps, "exps", torch.int8, n_e), _dev(term_signs, "term_signs", torch.int8, n_e),
        q, N, K, group, terms, batch,
        _dev(y, "y", torch.float32, batch * N), _stream(stream)), "sa_shiftadd_gemm_terms")


def sa_quantize_bcq(w: torch.Tensor, N: int, K: int, q: int, group: int, cycles: int,
                    signs: torch.Tensor, exps: torch.Tensor, stream=None) -> None:
    if group <= 0 or K % group:
        _check(SA_ERR_GROUP, "sa_quantize_bcq")
    _check(lib.sa_quantize_bcq(
        _dev(w, "w", torch.float32, N * K), N, K, q, group, cycles,
        _dev(signs, "signs", torch.int8, q * N * K),
        _dev(exps, "exps", torch.int8, q * N * (K // group)), _stream(stream)),
        "sa_quantize_bcq")


def sa_quantize_bcq_terms(w: torch.Tensor, N: int, K: int, q: int, group: int, cycles: int,
                          terms: int, signs: torch.Tensor, exps: torch.Tensor,
                          term_signs: torch.Tensor, stream=None) -> None:
    if group <= 0 or K % group:
        _check(SA_ERR_GROUP, "sa_quantize_bcq_terms")
    if terms < 1 or terms > SA_MAX_TERMS:
        _check(SA_ERR_SHAPE, "sa_quantize_bcq_terms")
    n_e = terms * q * N * (K // group)
    _check(lib.sa_quantize_bcq_terms(
        _dev(w, "w", torch.float32, N * K), N, K, q, group, cycles, terms,
        _dev(signs, "signs", torch.int8, q * N * K),
        _dev(exps, "exps", torch.int8, n_e), _dev(term_signs, "term_signs", torch.int8, n_e),
        _stream(stream)), "sa_quantize_bcq_terms")


def sa_gram_f16(x: torch.Tensor, K: int, T: int, H: torch.Tensor, stream=None) -> None:
    _check(lib.sa_gram_f16(_dev(x, "x", torch.float16, K * T), K, T,
                           _dev(H, "H", torch.float32, K * K), _stream(stream)), "sa_gram_f16")


def sa_inverse_cholesky_diag(H: torch.Tensor, K: int, damp: float, d: torch.Tensor,
                             workspace: torch.Tensor, stream=None) -> None:
    nbytes = workspace.numel() * workspace.element_size()
    _check(lib.sa_inverse_cholesky_diag(_dev(H, "H", torch.float32, K * K), K, float(damp),
                                        _dev(d, "d", torch.float64, K),
                                        _dev(workspace, "workspace", workspace.dtype,
                                             workspace.numel()), nbytes, _stream(stream)),
           "sa_inverse_cholesky_diag")


def sa_importance_criterion(w: torch.Tensor, N: int, K: int, d: torch.Tensor, out: torch.Tensor,
                            workspace: torch.Tensor, stream=None) -> None:
    nbytes = workspace.numel() * workspace.element_size()
    _check(lib.sa_importance_criterion(_dev(w, "w", torch.float32, N * K), N, K,
                                       _dev(d, "d", torch.float64, K),
                                       _dev(out, "out", torch.float64, 3),
                                       _dev(workspace, "workspace", workspace.dtype,
                                            workspace.numel()), nbytes, _stream(stream)),
           "sa_importance_criterion")


def sa_importance_criterion_noalloc(w: torch.Tensor, N: int, K: int, d: torch.Tensor,
                                    out: torch.Tensor, stream=None) -> None:
    _check(lib.sa_importance_criterion_noalloc(_dev(w, "w", torch.float32, N * K), N, K,
                                               _dev(d, "d", torch.float64, K),
                                               _dev(out, "out", torch.float64, 3),
                                               _stream(stream)),
           "sa_importance_criterion_noalloc")


def sa_fit_per_bit(c, errors, degree: int = 1):
    """Host: per-bit least-squares polynomial estimates ``[L][nb]`` (numpy in and out)."""
    import numpy as np
    c = np.ascontiguousarray(c, dtype=np.float64)
    errors = np.ascontiguousarray(errors, dtype=np.float64)
    L, nb = errors.shape
    out = np.empty((L, nb), dtype=np.float64)
    _check(lib.sa_fit_per_bit(c.ctypes.data, errors.ctypes.data, L, nb, degree, out.ctypes.data),
           "sa_fit_per_bit")
    return out


def sa_allocate_bits(cost, bits, budget: float):
    """Host: Eq. 4 -> ``(widths [L] int, objective)`` (numpy in and out)."""
    import numpy as np
    cost = np.ascontiguousarray(cost, dtype=np.float64)
    L, nb = cost.shape
    b = np.ascontiguousarray(bits, dtype=np.int32)
    out = np.empty(L, dtype=np.int32)
    obj = ctypes.c_double()
    _check(lib.sa_allocate_bits(cost.ctypes.data, b.ctypes.data, L, nb, float(budget),
                                out.ctypes.data, ctypes.byref(obj)), "sa_allocate_bits")
    return out, obj.value


def sa_read_probe(buf: torch.Tensor, nbytes: int, out: torch.Tensor, stream=None) -> None:
    """Plain read of ``nbytes`` bytes of ``buf`` (a measurement aid, see the header)."""
    if not isinstance(buf, torch.Tensor) or not buf.is_cuda:
        raise ValueError("buf must be a GPU tensor")
    if nbytes > buf.numel() * buf.element_size():
        raise ValueError("nbytes exceeds the buffer")
    _check(lib.sa_read_probe(buf.data_ptr(), nbytes,
                             _dev(out, "out", torch.float32, 256), _stream(stream)),
           "sa_read_probe")


# ------------------------------------------------------------------ conveniences

def quantize_bcq(w: torch.Tensor, q: int, group: int, cycles: int, stream=None):
    """``(signs int8 [q][N][K], exps int8 [q][N][K/group])`` of fp32 weights
    ``[N][K]`` (new device tensors), in the layer's format."""
    N, K = w.shape
    signs = torch.empty((q, N, K), dtype=torch.int8, device=w.device)
    exps = torch.empty((q, N, K // group), dtype=torch.int8, device=w.device)
    sa_quantize_bcq(w, N, K, q, group, cycles, signs, exps, stream)
    return signs, exps


def quantize_bcq_terms(w: torch.Tensor, q: int, group: int, cycles: int, terms: int,
                       stream=None):
    """``(signs [q][N][K], exps [q][N][K/group][terms], term_signs [q][N][K/group][terms])``
    (int8, new device tensors) with additive PoT scales."""
    N, K = w.shape
    signs = torch.empty((q, N, K), dtype=torch.int8, device=w.device)
    exps = torch.empty((q, N, K // group, terms), dtype=torch.int8, device=w.device)
    tsg = torch.empty((q, N, K // group, terms), dtype=torch.int8, device=w.device)
    sa_quantize_bcq_terms(w, N, K, q, group, cycles, terms, signs, exps, tsg, stream)
    return signs, exps, tsg


def pack_weights(signs: torch.Tensor, stream=None) -> torch.Tensor:
    """Packed planes of ``int8 [q][N][K]`` signs (a new uint8 device tensor)."""
    q, N, K = signs.shape
    packed = torch.empty(sa_packed_bytes(q, N, K), dtype=torch.uint8, device=signs.device)
    sa_pack_weights(signs, q, N, K, packed, stream)
    return packed


def shiftadd_gemm(x: torch.Tensor, packed_bits: torch.Tensor, exps: torch.Tensor, q: int, N: int,
                  K: int, group: int, out: Optional[torch.Tensor] = None,
                  stream=None) -> torch.Tensor:
    """``y = x W_q^T`` as a new (or the given) fp32 ``[batch][N]`` tensor."""
    batch = x.shape[0] if x.dim() == 2 else 1
    y = out if out is not None else torch.empty((batch, N), dtype=torch.float32, device=x.device)
    sa_shiftadd_gemm(x, packed_bits, exps, q, N, K, group, batch, y, stream)
    return y


def shiftadd_gemm_colwise(x: torch.Tensor, packed_bits: torch.Tensor, col_exps: torch.Tensor,
                          q: int, N: int, K: int, out: Optional[torch.Tensor] = None,
                          stream=None) -> torch.Tensor:
    """``y = x W_q^T`` with column-wise factors, as a new (or the given) fp32
    ``[batch][N]`` tensor."""
    batch = x.shape[0] if x.dim() == 2 else 1
    y = out if out is not None else torch.empty((batch, N), dtype=torch.float32, device=x.device)
    sa_shiftadd_gemm_colwise(x, packed_bits, col_exps, q, N, K, batch, y, stream)
    return y


def shiftadd_gemm_blockwise(x: torch.Tensor, packed_bits: torch.Tensor, blk_exps: torch.Tensor,
                            q: int, N: int, K: int, row_block: int,
                            out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """``y = x W_q^T`` with block-wise factors, as a new (or the given) fp32
    ``[batch][N]`` tensor."""
    batch = x.shape[0] if x.dim() == 2 else 1
    y = out if out is not None else torch.empty((batch, N), dtype=torch.float32, device=x.device)
    sa_shiftadd_gemm_blockwise(x, packed_bits, blk_exps, q, N, K, row_block, batch, y, stream)
    return y


def bit_criterion(w: torch.Tensor, x: torch.Tensor, damp: float = 0.01, stream=None):
    """Eq. 3 for one layer: ``(C, ||IS||_F, STD(IS), d)`` from fp32 weights
    ``[N][K]`` and fp16 calibration activations ``[K][T]`` on the device
    (workspaces are new device tensors)."""
    N, K = w.shape
    T = x.shape[1]
    H = torch.empty((K, K), dtype=torch.float32, device=w.device)
    sa_gram_f16(x, K, T, H, stream)
    d = torch.empty(K, dtype=torch.float64, device=w.device)
    ws = torch.empty(lib.sa_inverse_cholesky_workspace(K), dtype=torch.uint8, device=w.device)
    sa_inverse_cholesky_diag(H, K, damp, d, ws, stream)
    out = torch.empty(3, dtype=torch.float64, device=w.device)
    ws2 = torch.empty(lib.sa_importance_workspace(), dtype=torch.uint8, device=w.device)
    sa_importance_criterion(w, N, K, d, out, ws2, stream)
    o = out.cpu()
    return float(o[0]), float(o[1]), float(o[2]), d
