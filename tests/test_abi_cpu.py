"""The C ABI on the CPU: the library loads, exports every declared symbol, and
rejects invalid arguments on the host before any HIP call.  No compute call is
made here (there is no GPU in this environment)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "shiftadd.h")

sa = pytest.importorskip("paper_2406_05981_amd.shiftadd",
                         reason="libshiftadd.so not built (python -m paper_2406_05981_amd.build)")
from tests import _layout  # noqa: E402

A = 1 << 20  # a non-null, 16-byte aligned fake address; never dereferenced here


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"SA_API\s+[\w\s\*]+?\b(sa_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_symbols()
    assert {"sa_pack_weights", "sa_unpack_weights", "sa_build_lut", "sa_shiftadd_gemm",
            "sa_packed_bytes", "sa_packed_offset", "sa_plan_gemm", "sa_status_string",
            "sa_version"} <= set(names)
    raw = ctypes.CDLL(sa.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n


def test_version_and_status_strings():
    assert "gfx950" in sa.sa_version()
    for st in range(0, -7, -1):
        assert sa.sa_status_string(st) not in ("", "unknown status")
    assert sa.sa_status_string(-99) == "unknown status"


def test_packed_bytes():
    assert sa.sa_packed_bytes(3, 4096, 4096) == 3 * 4096 * 512
    assert sa.sa_packed_bytes(0, 8, 8) == 0
    assert sa.sa_packed_bytes(9, 8, 8) == 0
    assert sa.sa_packed_bytes(1, 8, 12) == 0


@pytest.mark.parametrize("q,N,K", [(1, 1, 8), (2, 65, 136), (3, 64, 128), (2, 130, 264),
                                   (1, 200, 1040), (3, 5, 256)])
def test_layout_is_a_bijection_and_matches_restatement(q, N, K):
    off = _layout.offsets(q, N, K)
    assert np.array_equal(np.sort(off.reshape(-1)), np.arange(q * N * (K // 8)))
    rng = np.random.default_rng(0)
    for _ in range(200):
        i, n, c = int(rng.integers(q)), int(rng.integers(N)), int(rng.integers(K // 8))
        assert sa.sa_packed_offset(q, N, K, i, n, c) == off[i, n, c]
    assert sa.sa_packed_offset(q, N, K, q, 0, 0) == -1
    assert sa.sa_packed_offset(q, N, K, 0, N, 0) == -1
    assert sa.sa_packed_offset(q, N, K, 0, 0, K // 8) == -1


def test_layout_tiles_are_contiguous_16_byte_rows():
    """A 64-row tile of a full 16-chunk block is 1 KiB, 16 bytes per row, and
    position p of row r holds chunk (p + r) mod 16."""
    q, N, K = 1, 128, 256
    off = _layout.offsets(q, N, K)
    for r in (0, 1, 17, 63):
        row = off[0, r, :16]
        assert sorted(row.tolist()) == list(range(16 * r, 16 * r + 16))
        for c in range(16):
            assert row[c] - 16 * r == (c - r) % 16


def _gemm(x=A, p=A, e=A, q=3, N=64, K=256, G=128, B=1, y=A):
    return sa.lib.sa_shiftadd_gemm(x, p, e, q, N, K, G, B, y, None)


def test_gemm_validation_codes():
    assert _gemm(x=None) == sa.SA_ERR_NULL
    assert _gemm(p=None) == sa.SA_ERR_NULL
    assert _gemm(e=None) == sa.SA_ERR_NULL
    assert _gemm(y=None) == sa.SA_ERR_NULL
    assert _gemm(q=0) == sa.SA_ERR_Q
    assert _gemm(q=9) == sa.SA_ERR_Q
    assert _gemm(N=0) == sa.SA_ERR_SHAPE
    assert _gemm(K=12) == sa.SA_ERR_SHAPE
    assert _gemm(K=0) == sa.SA_ERR_SHAPE
    assert _gemm(B=0) == sa.SA_ERR_SHAPE
    assert _gemm(B=sa.SA_MAX_BATCH + 1) == sa.SA_ERR_SHAPE
    # one plane of packed keys must stay below 2^31 bytes
    assert sa.sa_packed_bytes(1, 1 << 17, 1 << 17) == 0
    assert sa.sa_packed_bytes(1, (1 << 17) - 1, 1 << 17) == ((1 << 17) - 1) * (1 << 14)
    assert _gemm(G=0) == sa.SA_ERR_GROUP
    assert _gemm(G=12) == sa.SA_ERR_GROUP
    assert _gemm(G=96) == sa.SA_ERR_GROUP  # 256 % 96 != 0
    assert _gemm(x=A + 8) == sa.SA_ERR_ALIGN
    assert _gemm(p=A + 4) == sa.SA_ERR_ALIGN
    assert _gemm(y=A + 2) == sa.SA_ERR_ALIGN
    assert _gemm(e=A + 1, x=None) == sa.SA_ERR_NULL  # exps may be unaligned; NULL x still caught


def test_pack_lut_validation_codes():
    L = sa.lib
    assert L.sa_pack_weights(None, 1, 8, 8, A, None) == sa.SA_ERR_NULL
    assert L.sa_pack_weights(A, 1, 8, 8, None, None) == sa.SA_ERR_NULL
    assert L.sa_pack_weights(A, 0, 8, 8, A, None) == sa.SA_ERR_Q
    assert L.sa_pack_weights(A, 1, 8, 9, A, None) == sa.SA_ERR_SHAPE
    assert L.sa_pack_weights(A, 1, 8, 8, A + 1, None) == sa.SA_ERR_ALIGN
    assert L.sa_unpack_weights(None, 1, 8, 8, A, None) == sa.SA_ERR_NULL
    assert L.sa_unpack_weights(A, 1, -1, 8, A, None) == sa.SA_ERR_SHAPE
    assert L.sa_build_lut(None, 8, 1, A, None) == sa.SA_ERR_NULL
    assert L.sa_build_lut(A, 10, 1, A, None) == sa.SA_ERR_SHAPE
    assert L.sa_build_lut(A, 8, 0, A, None) == sa.SA_ERR_SHAPE
    assert L.sa_build_lut(A + 2, 8, 1, A, None) == sa.SA_ERR_ALIGN


def test_f16_output_validation():
    L = sa.lib
    f = L.sa_shiftadd_gemm_f16
    assert f(A, A, A, 3, 100, 1024, 128, 1, None, None) == sa.SA_ERR_NULL
    assert f(A, A, A, 9, 100, 1024, 128, 1, A, None) == sa.SA_ERR_Q
    assert f(A, A, A, 3, 100, 1024, 100, 1, A, None) == sa.SA_ERR_GROUP
    assert f(A, A, A, 3, 100, 1024, 128, 0, A, None) == sa.SA_ERR_SHAPE
    assert f(A, A, A, 3, 100, 1024, 128, 1, A + 2, None) == sa.SA_ERR_ALIGN


def test_kslice_validation():
    L = sa.lib
    E = sa
    assert sa.sa_kslice_workspace_bytes(100, 2048) == 4 * 2 * 100
    assert sa.sa_kslice_workspace_bytes(100, 1536) == 0
    assert sa.sa_kslice_workspace_bytes(0, 2048) == 0
    ws = 4 * 2 * 100
    f = L.sa_shiftadd_gemm_kslice
    assert f(A, A, A, 3, 100, 2048, 128, A, None, ws, None) == E.SA_ERR_NULL
    assert f(A, A, None, 3, 100, 2048, 128, A, A, ws, None) == E.SA_ERR_NULL
    assert f(A, A, A, 9, 100, 2048, 128, A, A, ws, None) == E.SA_ERR_Q
    assert f(A, A, A, 3, 100, 1536, 128, A, A, ws, None) == E.SA_ERR_SHAPE
    assert f(A, A, A, 3, 100, 2048, 64, A, A, ws, None) == E.SA_ERR_GROUP
    assert f(A, A, A, 3, 100, 2048, 100, A, A, ws, None) == E.SA_ERR_GROUP
    assert f(A, A, A, 3, 100, 2048, 128, A, A, ws - 4, None) == E.SA_ERR_SHAPE
    assert f(A + 2, A, A, 3, 100, 2048, 128, A, A, ws, None) == E.SA_ERR_ALIGN
    assert f(A, A, A, 3, 100, 2048, 128, A + 4, A, ws, None) == E.SA_ERR_ALIGN
    assert f(A, A, A, 3, 100, 2048, 128, A, A + 2, ws, None) == E.SA_ERR_ALIGN


def test_plans():
    p = sa.sa_plan_gemm(3, 4096, 4096, 128, 1)
    assert p["path"] == 1 and p["rows_per_wg"] == 16 and p["workgroups"] == 256
    assert p["pieces"] == 1 and p["lds_bytes"] <= 80 * 1024
    assert sa.sa_plan_gemm(3, 100, 256, 8, 2)["path"] == 0
    assert sa.sa_plan_gemm(3, 100, 768, 768, 1)["path"] == 1
    assert sa.sa_plan_gemm(3, 100, 768, 768, 2)["path"] == 2
    assert sa.sa_plan_gemm(3, 8192, 28672, 128, 1)["pieces"] == 7
    # batch kernel: 1024-column pieces, one workgroup per (row tile, group of 4
    # batch rows), grid padded to whole rounds of 8 workgroups per XCD
    big = sa.sa_plan_gemm(3, 28672, 8192, 128, 8)
    assert big["path"] == 2 and big["pieces"] == 8 and big["rows_per_wg"] == 64
    assert big["workgroups"] == 8 * 2 * ((28672 // 64 + 7) // 8)
    assert big["lds_bytes"] <= 80 * 1024
    # every row-tile height of the batch kernel is reachable
    # (shapes of the GPU parity list)
    heights = {sa.sa_plan_gemm(*c)["rows_per_wg"] for c in
               [(2, 300, 384, 128, 2), (3, 4100, 384, 384, 13), (1, 28672, 1152, 128, 5)]}
    assert heights == {16, 32, 64}
    with pytest.raises(sa.SaError):
        sa.sa_plan_gemm(3, 100, 256, 24, 1)


def test_read_probe_validation_codes():
    f = sa.lib.sa_read_probe
    assert f(None, 1024, A, None) == sa.SA_ERR_NULL
    assert f(A, 1024, None, None) == sa.SA_ERR_NULL
    assert f(A, 0, A, None) == sa.SA_ERR_SHAPE
    assert f(A, 1000, A, None) == sa.SA_ERR_SHAPE  # not a multiple of 16
    assert f(A, (1 << 40) + 16, A, None) == sa.SA_ERR_SHAPE
    assert f(A + 8, 1024, A, None) == sa.SA_ERR_ALIGN


def test_quantize_validation_codes():
    f = sa.lib.sa_quantize_bcq

    def call(w=A, N=16, K=256, q=3, G=128, T=2, s=A, e=A):
        return f(w, N, K, q, G, T, s, e, None)

    assert call(w=None) == sa.SA_ERR_NULL
    assert call(s=None) == sa.SA_ERR_NULL
    assert call(e=None) == sa.SA_ERR_NULL
    assert call(q=0) == sa.SA_ERR_Q
    assert call(q=9) == sa.SA_ERR_Q
    assert call(N=0) == sa.SA_ERR_SHAPE
    assert call(K=12) == sa.SA_ERR_SHAPE
    assert call(G=0) == sa.SA_ERR_GROUP
    assert call(G=12) == sa.SA_ERR_GROUP
    assert call(G=96) == sa.SA_ERR_GROUP   # 256 % 96 != 0
    assert call(T=-1) == sa.SA_ERR_SHAPE
    assert call(T=sa.SA_MAX_CYCLES + 1) == sa.SA_ERR_SHAPE
    assert call(w=A + 2) == sa.SA_ERR_ALIGN
    assert call(w=A + 8) == sa.SA_ERR_ALIGN   # 16-byte loads
    assert call(s=A + 4) == sa.SA_ERR_ALIGN   # 8-byte stores
    assert call(e=A + 1, w=None) == sa.SA_ERR_NULL  # exps may be unaligned


def test_colwise_validation_codes():
    f = sa.lib.sa_shiftadd_gemm_colwise

    def call(x=A, p=A, e=A, q=3, N=64, K=256, B=1, y=A):
        return f(x, p, e, q, N, K, B, y, None)

    assert call(x=None) == sa.SA_ERR_NULL
    assert call(p=None) == sa.SA_ERR_NULL
    assert call(e=None) == sa.SA_ERR_NULL
    assert call(y=None) == sa.SA_ERR_NULL
    assert call(q=0) == sa.SA_ERR_Q
    assert call(q=9) == sa.SA_ERR_Q
    assert call(K=200) == sa.SA_ERR_SHAPE   # K % 128 != 0
    assert call(K=12) == sa.SA_ERR_SHAPE
    assert call(B=0) == sa.SA_ERR_SHAPE
    assert call(B=sa.SA_MAX_BATCH + 1) == sa.SA_ERR_SHAPE
    assert call(x=A + 8) == sa.SA_ERR_ALIGN
    assert call(p=A + 4) == sa.SA_ERR_ALIGN
    assert call(y=A + 4) == sa.SA_ERR_ALIGN
    assert call(e=A + 4) == sa.SA_ERR_ALIGN
    p = sa.sa_plan_gemm_colwise(3, 4096, 4096, 1)
    assert p["path"] == 3 and p["workgroups"] == 256 and p["pieces"] == 1
    assert sa.sa_plan_gemm_colwise(3, 8192, 28672, 1)["pieces"] == 7
    p = sa.sa_plan_gemm_colwise(3, 4096, 4096, 16)  # the batch kernel, one build per plane
    assert p["path"] == 6 and p["rows_per_wg"] == 64
    # several pieces and at most one workgroup per CU: 16 waves, two pieces at once
    assert sa.sa_plan_gemm(3, 4096, 11008, 128, 1)["threads"] == 1024
    assert sa.sa_plan_gemm(4, 3584, 8192, 128, 1)["threads"] == 1024
    assert sa.sa_plan_gemm(5, 4096, 11008, 128, 1)["threads"] == 512   # registers
    # 449..512 row groups and several pieces: two groups per workgroup, 16 waves
    p = sa.sa_plan_gemm(3, 8192, 28672, 128, 1)
    assert p["threads"] == 1024 and p["workgroups"] == 256 and p["rows_per_wg"] == 32
    assert sa.sa_plan_gemm(3, 28672, 8192, 128, 1)["threads"] == 512   # 1792 groups
    assert sa.sa_plan_gemm(3, 4200, 8320, 128, 1)["workgroups"] == 263  # 263 groups: one each
    assert sa.sa_plan_gemm(3, 4096, 4096, 128, 1)["threads"] == 512    # one piece
    assert sa.sa_plan_gemm_colwise(3, 4096, 11008, 1)["threads"] == 1024
    assert sa.sa_plan_gemm_blockwise(3, 4096, 11008, 512, 1)["threads"] == 1024
    assert sa.sa_plan_gemm_blockwise(4, 4096, 11008, 512, 1)["threads"] == 512
    with pytest.raises(sa.SaError):
        sa.sa_plan_gemm_colwise(3, 100, 200, 1)


def test_blockwise_validation_codes():
    f = sa.lib.sa_shiftadd_gemm_blockwise

    def call(x=A, p=A, e=A, q=3, N=64, K=256, rb=8, B=1, y=A):
        return f(x, p, e, q, N, K, rb, B, y, None)

    assert call(x=None) == sa.SA_ERR_NULL
    assert call(p=None) == sa.SA_ERR_NULL
    assert call(e=None) == sa.SA_ERR_NULL
    assert call(y=None) == sa.SA_ERR_NULL
    assert call(q=0) == sa.SA_ERR_Q
    assert call(q=9) == sa.SA_ERR_Q
    assert call(K=200) == sa.SA_ERR_SHAPE
    assert call(rb=0) == sa.SA_ERR_SHAPE
    assert call(B=0) == sa.SA_ERR_SHAPE
    assert call(x=A + 8) == sa.SA_ERR_ALIGN
    assert call(e=A + 8) == sa.SA_ERR_ALIGN
    assert call(y=A + 4) == sa.SA_ERR_ALIGN
    p = sa.sa_plan_gemm_blockwise(3, 4096, 4096, 512, 1)
    assert p["path"] == 4 and p["workgroups"] == 256
    p = sa.sa_plan_gemm_blockwise(3, 4096, 4096, 512, 16)  # the batch kernel
    assert p["path"] == 5 and p["rows_per_wg"] == 64 and p["workgroups"] == 256
    with pytest.raises(sa.SaError):
        sa.sa_plan_gemm_blockwise(3, 4096, 4096, 0, 1)


def test_terms_validation_codes():
    f = sa.lib.sa_shiftadd_gemm_terms

    def call(x=A, p=A, e=A, s=A, q=3, N=64, K=256, G=128, T=2, B=1, y=A):
        return f(x, p, e, s, q, N, K, G, T, B, y, None)

    assert call(s=None) == sa.SA_ERR_NULL
    assert call(e=None) == sa.SA_ERR_NULL
    assert call(x=None) == sa.SA_ERR_NULL
    assert call(q=9) == sa.SA_ERR_Q
    assert call(G=64) == sa.SA_ERR_GROUP    # the row kernel takes groups of 128 columns
    assert call(G=96) == sa.SA_ERR_GROUP
    assert call(T=0) == sa.SA_ERR_SHAPE
    assert call(T=sa.SA_MAX_TERMS + 1) == sa.SA_ERR_SHAPE
    assert call(x=A + 8) == sa.SA_ERR_ALIGN


def test_quantize_terms_validation_codes():
    f = sa.lib.sa_quantize_bcq_terms

    def call(w=A, N=16, K=256, q=3, G=128, T=2, n=2, s=A, e=A, t=A):
        return f(w, N, K, q, G, T, n, s, e, t, None)

    assert call(t=None) == sa.SA_ERR_NULL
    assert call(w=None) == sa.SA_ERR_NULL
    assert call(n=0) == sa.SA_ERR_SHAPE
    assert call(n=sa.SA_MAX_TERMS + 1) == sa.SA_ERR_SHAPE
    assert call(q=9) == sa.SA_ERR_Q
    assert call(G=96) == sa.SA_ERR_GROUP
    assert call(w=A + 8) == sa.SA_ERR_ALIGN


def test_alloc_validation_codes():
    L = sa.lib
    assert L.sa_gram_f16(None, 128, 32, A, None) == sa.SA_ERR_NULL
    assert L.sa_gram_f16(A, 192, 32, A, None) == sa.SA_ERR_SHAPE     # K % 128
    assert L.sa_gram_f16(A, 128, 40, A, None) == sa.SA_ERR_SHAPE     # T % 32
    assert L.sa_gram_f16(A + 8, 128, 32, A, None) == sa.SA_ERR_ALIGN
    ws = L.sa_inverse_cholesky_workspace(64)
    assert ws >= 64 * 64 * 8
    assert L.sa_inverse_cholesky_diag(A, 64, 0.01, A, None, ws, None) == sa.SA_ERR_NULL
    assert L.sa_inverse_cholesky_diag(A, 64, 0.01, A, A, ws - 1, None) == sa.SA_ERR_SHAPE
    assert L.sa_inverse_cholesky_diag(A, 64, -1.0, A, A, ws, None) == sa.SA_ERR_SHAPE
    assert L.sa_inverse_cholesky_diag(A, 64, 0.01, A, A + 8, ws, None) == sa.SA_ERR_ALIGN
    w2 = L.sa_importance_workspace()
    assert L.sa_importance_criterion(A, 4, 64, A, A, A, w2 - 8, None) == sa.SA_ERR_SHAPE
    assert L.sa_importance_criterion(A, 0, 64, A, A, A, w2, None) == sa.SA_ERR_SHAPE
