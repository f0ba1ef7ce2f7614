"""GPU parity of the layer with column-wise factors (sa_shiftadd_gemm_colwise,
"Ours (Acc.)") against the CPU oracle (oracle.shiftadd_gemm_colwise).

Bar (fixed here): max |y - y_ref| / sum|terms| <= 2e-3 per output, with the
same stricter 1e-5 alarm as the row-wise layer: the activations are shifted
exactly in fp32 and the tables are fp32, so the error is fp32 rounding of the
table sums and the accumulation.
"""
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


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def run(c, packed=None):
    q, N, K, B = c["q"], c["N"], c["K"], c["B"]
    if packed is None:
        packed = sa.pack_weights(dev(c["signs"]))
    y = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm_colwise(dev(c["x"]), packed, dev(c["col_exps"]), q, N, K, B, y)
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


def check(y, y_ref, a_ref, what):
    assert np.isfinite(y).all(), what
    err = np.abs(y - y_ref)
    zero = a_ref == 0
    assert (err[zero] == 0).all(), what
    worst = float((err[~zero] / a_ref[~zero]).max()) if (~zero).any() else 0.0
    say(f"  {what}: max |y-y_ref|/sum|terms| = {worst:.3e}")
    assert worst <= TOL and worst <= ALARM, what


CASES = [
    # (q, N, K, B, label)
    (3, 768, 768, 1, "one piece, one row group per workgroup"),
    (2, 130, 384, 1, "ragged row count"),
    (1, 33, 128, 3, "one block, batch 3"),
    (4, 4100, 1024, 2, "several row groups per workgroup"),
    (3, 64, 8192, 1, "two pieces"),
    (8, 17, 256, 1, "eight planes"),
    (3, 300, 4224, 4, "ragged last piece (33 blocks)"),
    (2, 1000, 2048, 16, "batch 16"),
    (3, 1000, 8320, 1, "16 waves, three pieces, one-block last piece"),
    (2, 4096, 8192, 1, "16 waves, 256 workgroups"),
    (3, 8000, 8320, 1, "16 waves, two row groups per workgroup"),
]


@pytest.mark.parametrize("q,N,K,B,label", CASES, ids=[c[-1] for c in CASES])
def test_colwise_parity(q, N, K, B, label):
    say(f"colwise q={q} N={N} K={K} B={B}: {label}")
    c = workloads.colwise_case(q, N, K, B, seed=q + N + K + B)
    y = run(c)
    y_ref, a_ref = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"])
    check(y, y_ref, a_ref, label)


def test_colwise_exponent_extremes_and_zero_rows():
    """Exponents at +-30 with large and tiny activations (shifts stay exact in
    fp32), a zero activation row, and planes whose signs are all +1 / all -1."""
    q, N, K, B = 3, 96, 512, 3
    c = workloads.colwise_case(q, N, K, B, seed=9, exp_range=(-30, 30))
    x = c["x"].astype(np.float32)
    x[1] = 0.0
    x[2, ::7] = 60000.0
    x[2, 3::7] = 6e-8            # fp16 subnormals
    c["x"] = x.astype(np.float16)
    c["signs"][0, :8] = 1
    c["signs"][1, 8:16] = -1
    say("colwise extremes")
    y = run(c)
    y_ref, a_ref = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"])
    check(y, y_ref, a_ref, "exponents +-30, zero row, subnormals")
    assert (y[1] == 0).all()


def test_colwise_constant_columns_match_row_wise_kernel():
    """With one exponent per plane for every column, the column-wise layer is
    the row-wise layer with G = K (a different kernel path): both within the
    bar of the oracle and of each other."""
    q, N, K, B = 3, 512, 2048, 1
    c = workloads.colwise_case(q, N, K, B, seed=11)
    c["col_exps"][:] = c["col_exps"][:, :1]
    y = run(c)
    exps = np.broadcast_to(c["col_exps"][:, None, :1], (q, N, 1)).copy()
    yr = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm(dev(c["x"]), sa.pack_weights(dev(c["signs"])), dev(exps), q, N, K, K,
                        B, yr)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], exps, K)
    check(y, y_ref, a_ref, "column-wise kernel, constant columns")
    check(yr.cpu().numpy().astype(np.float64), y_ref, a_ref, "row-wise kernel, G = K")


@pytest.mark.parametrize("N,K", [(4096, 4096), (11008, 4096), (4096, 11008)])
def test_colwise_full_size_sampled(N, K):
    """LLaMA-2-7B projection shapes, q = 3, batch 1, in the launch configuration
    the benchmark times; 512 sampled rows compared with the oracle."""
    q, B = 3, 1
    say(f"colwise full size N={N} K={K}")
    c = workloads.colwise_case(q, N, K, B, seed=1)
    y = run(c)
    rows = np.sort(np.random.default_rng(0).choice(N, 512, replace=False))
    rows[-1] = N - 1
    y_ref, a_ref = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"], rows=rows)
    check(y[:, rows], y_ref, a_ref, f"{N}x{K} sampled")


def test_colwise_error_codes():
    c = workloads.colwise_case(2, 64, 256, 1, seed=1)
    packed = sa.pack_weights(dev(c["signs"]))
    y = torch.empty((1, 64), dtype=torch.float32, device="cuda")
    c200 = workloads.colwise_case(2, 64, 200, 1, seed=1)
    with pytest.raises(sa.SaError):  # K % 128 != 0
        sa.sa_shiftadd_gemm_colwise(dev(c200["x"]), sa.pack_weights(dev(c200["signs"])),
                                    dev(c200["col_exps"]), 2, 64, 200, 1, y)
    with pytest.raises(sa.SaError):
        sa.sa_shiftadd_gemm_colwise(dev(c["x"]), packed, dev(c["col_exps"]), 9, 64, 256, 1, y)


# Batch >= 2 runs the batch kernel (plan path 6): each plane's tables are built
# in turn from the shifted activations; 16, 32 or 64 rows per workgroup.
BATCH_CASES = [
    # (q, N, K, B, label)
    (3, 1000, 1024, 8, "KW=1, two quads"),
    (3, 4096, 1024, 8, "KW=2"),
    (4, 4096, 512, 16, "KW=4, four planes"),
    (8, 2048, 512, 16, "eight planes"),
    (2, 130, 384, 5, "ragged quad and rows"),
    (1, 77, 4224, 6, "one plane, ragged last piece"),
    (5, 300, 2048, 13, "five planes, two pieces, ragged quad"),
]


@pytest.mark.parametrize("q,N,K,B,label", BATCH_CASES, ids=[c[-1] for c in BATCH_CASES])
def test_colwise_batch_parity(q, N, K, B, label):
    plan = sa.sa_plan_gemm_colwise(q, N, K, B)
    assert plan["path"] == 6
    say(f"colwise batch q={q} N={N} K={K} B={B} rows/wg={plan['rows_per_wg']}: {label}")
    c = workloads.colwise_case(q, N, K, B, seed=q + N + K + B)
    y = run(c)
    y_ref, a_ref = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"])
    check(y, y_ref, a_ref, label)


def test_colwise_batch_rows_agree_with_batch_one():
    """Batch rows of the batch kernel against the row kernel on each row alone."""
    q, N, K, B = 3, 1024, 2048, 8
    c = workloads.colwise_case(q, N, K, B, seed=5)
    packed = sa.pack_weights(dev(c["signs"]))
    y = run(c, packed)
    y_ref, a_ref = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"])
    check(y, y_ref, a_ref, "batch 8")
    for b in (0, 3, 7):
        y1 = run(dict(c, B=1, x=c["x"][b:b + 1]), packed)
        check(y1, y_ref[b:b + 1], a_ref[b:b + 1], f"batch row {b} alone")


@pytest.mark.parametrize("N,K", [(4096, 4096), (11008, 4096)])
def test_colwise_batch_full_size_sampled(N, K):
    q, B = 3, 16
    say(f"colwise batch full size N={N} K={K} B={B}")
    c = workloads.colwise_case(q, N, K, B, seed=2)
    y = run(c)
    rows = np.sort(np.random.default_rng(1).choice(N, 256, replace=False))
    rows[-1] = N - 1
    y_ref, a_ref = oracle.shiftadd_gemm_colwise(c["x"], c["signs"], c["col_exps"], rows=rows)
    check(y[:, rows], y_ref, a_ref, f"{N}x{K} batch {B} sampled")
