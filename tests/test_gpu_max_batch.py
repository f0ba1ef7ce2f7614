"""GPU parity at the largest batch the boundary accepts (SA_MAX_BATCH = 256, 64
quads of the batch kernel) for every layer entry point, against the CPU oracle.

Bar (fixed here, as for the layer): max |y - y_ref| / sum|terms| <= 2e-3 per
output, with the 1e-5 alarm of fp32 tables."""
import sys

import numpy as np
import pytest

import oracle
import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - CPU-only environment
    pytest.skip("no GPU", allow_module_level=True)
sa = pytest.importorskip("paper_2406_05981_amd.shiftadd")

TOL = 2e-3
ALARM = 1e-5
B = sa.SA_MAX_BATCH


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def out(N):
    return torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")


def check(y, y_ref, a_ref, what):
    y = y.cpu().numpy().astype(np.float64)
    assert y.shape == y_ref.shape, what
    assert np.isfinite(y).all(), what
    err = np.abs(y - y_ref)
    zero = a_ref == 0
    assert (err[zero] == 0).all(), what
    worst = float((err[~zero] / a_ref[~zero]).max()) if (~zero).any() else 0.0
    say(f"  {what}: max |y-y_ref|/sum|terms| = {worst:.3e}")
    assert worst <= TOL and worst <= ALARM, what


@pytest.mark.parametrize("q,N,K,G", [(2, 130, 1152, 128), (3, 70, 4096, 128), (2, 33, 200, 40)],
                         ids=["batch kernel", "batch kernel, 4 pieces", "generic kernel"])
def test_row_wise_max_batch(q, N, K, G):
    say(f"row-wise q={q} N={N} K={K} G={G} B={B} path={sa.sa_plan_gemm(q, N, K, G, B)['path']}")
    c = workloads.random_case(q, N, K, G, B, seed=41, exp_range=(-10, -2))
    y = out(N)
    sa.sa_shiftadd_gemm(dev(c["x"]), sa.pack_weights(dev(c["signs"])), dev(c["exps"]), q, N, K, G,
                        B, y)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], G)
    check(y, y_ref, a_ref, "row-wise")


@pytest.mark.parametrize("q,N,K,T", [(2, 100, 1024, 3), (3, 70, 4096, 2)],
                         ids=["per-piece loads", "preloaded exponents"])
def test_terms_max_batch(q, N, K, T):
    say(f"terms q={q} N={N} K={K} T={T} B={B}")
    c = workloads.terms_case(q, N, K, 128, B, T, seed=42)
    y = out(N)
    sa.sa_shiftadd_gemm_terms(dev(c["x"]), sa.pack_weights(dev(c["signs"])), dev(c["exps"]),
                              dev(c["term_signs"]), q, N, K, 128, T, B, y)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], 128)
    check(y, y_ref, a_ref, "additive")


def test_colwise_max_batch():
    q, N, K = 3, 90, 1280
    say(f"colwise q={q} N={N} K={K} B={B}")
    c = workloads.colwise_case(q, N, K, B, seed=43)
    y = out(N)
    sa.sa_shiftadd_gemm_colwise(dev(c["x"]), sa.pack_weights(dev(c["signs"])), dev(c["col_exps"]),
                                q, N, K, B, y)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"])
    check(y, y_ref, a_ref, "column-wise")


@pytest.mark.parametrize("rb", [64, 23], ids=["scalar exponent loads", "per-lane exponent loads"])
def test_blockwise_max_batch(rb):
    q, N, K = 3, 128, 1024
    plan = sa.sa_plan_gemm_blockwise(q, N, K, rb, B)
    say(f"blockwise q={q} N={N} K={K} B={B} row_block={rb} rows/wg={plan['rows_per_wg']}")
    c = workloads.blockwise_case(q, N, K, B, rb, seed=44)
    y = out(N)
    sa.sa_shiftadd_gemm_blockwise(dev(c["x"]), sa.pack_weights(dev(c["signs"])),
                                  dev(c["blk_exps"]), q, N, K, rb, B, y)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb)
    check(y, y_ref, a_ref, "block-wise")
