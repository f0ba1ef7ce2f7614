"""GPU parity of the layer with block-wise factors (sa_shiftadd_gemm_blockwise,
"Ours (Lat.)") against the CPU oracle (oracle.shiftadd_gemm_blockwise).

Bar (fixed here): max |y - y_ref| / sum|terms| <= 2e-3 per output, with the
stricter 1e-5 alarm of the fp32 tables: each queried fp32 entry is shifted
exactly (ldexp) before it is added.
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


def run(c):
    q, N, K, B, rb = c["q"], c["N"], c["K"], c["B"], c["row_block"]
    packed = sa.pack_weights(dev(c["signs"]))
    y = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm_blockwise(dev(c["x"]), packed, dev(c["blk_exps"]), q, N, K, rb, B, y)
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
    # (q, N, K, B, row_block, label)
    (3, 768, 768, 1, 96, "N/8-row blocks, one piece"),
    (2, 130, 384, 1, 17, "ragged rows, 17-row blocks (not a multiple of 16)"),
    (1, 33, 128, 3, 1, "a factor per row, batch 3"),
    (4, 4100, 1024, 2, 513, "several row groups per workgroup"),
    (3, 64, 8192, 1, 8, "two pieces, 8-row blocks"),
    (8, 17, 256, 1, 17, "eight planes, one block of rows"),
    (3, 300, 4224, 4, 40, "ragged last piece (33 blocks), batch 4"),
    (5, 200, 1024, 2, 25, "five planes"),
    (3, 1000, 8320, 1, 125, "16 waves, three pieces, one-block last piece"),
    (2, 4096, 8192, 1, 512, "16 waves, 256 workgroups"),
    (3, 8000, 8320, 1, 1000, "16 waves, two row groups per workgroup"),
    (4, 1000, 8320, 1, 125, "four planes: 8 waves"),
]


@pytest.mark.parametrize("q,N,K,B,rb,label", CASES, ids=[c[-1] for c in CASES])
def test_blockwise_parity(q, N, K, B, rb, label):
    say(f"blockwise q={q} N={N} K={K} B={B} row_block={rb}: {label}")
    c = workloads.blockwise_case(q, N, K, B, rb, seed=q + N + K + B + rb)
    y = run(c)
    y_ref, a_ref = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb)
    check(y, y_ref, a_ref, label)


def test_blockwise_exponent_extremes():
    q, N, K, B, rb = 3, 96, 512, 3, 12
    c = workloads.blockwise_case(q, N, K, B, rb, seed=9, exp_range=(-30, 30))
    x = c["x"].astype(np.float32)
    x[1] = 0.0
    x[2, ::7] = 60000.0
    x[2, 3::7] = 6e-8
    c["x"] = x.astype(np.float16)
    say("blockwise extremes")
    y = run(c)
    y_ref, a_ref = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb)
    check(y, y_ref, a_ref, "exponents +-30, zero row, subnormals")
    assert (y[1] == 0).all()


def test_blockwise_constant_blocks_match_row_wise_kernel():
    """Block exponents equal over each 128-column block and over 16-row blocks:
    the layer is then the row-wise layer with G = 128 (another kernel path)."""
    q, N, K, B, rb = 3, 512, 2048, 1, 16
    c = workloads.blockwise_case(q, N, K, B, rb, seed=11)
    e = c["blk_exps"]
    e[:] = e[:, :, ::16].repeat(16, axis=2)
    y = run(c)
    exps = np.repeat(e[:, :, ::16], rb, axis=1)[:, :N]
    yr = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm(dev(c["x"]), sa.pack_weights(dev(c["signs"])), dev(exps), q, N, K, 128,
                        B, yr)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], exps, 128)
    check(y, y_ref, a_ref, "block-wise kernel, constant blocks")
    check(yr.cpu().numpy().astype(np.float64), y_ref, a_ref, "row-wise kernel, G = 128")


@pytest.mark.parametrize("N,K", [(4096, 4096), (11008, 4096), (4096, 11008)])
def test_blockwise_full_size_sampled(N, K):
    """LLaMA-2-7B projection shapes, q = 3, batch 1, row_block = N / 8, in the
    launch configuration the benchmark times; 512 sampled rows."""
    q, B, rb = 3, 1, N // 8
    say(f"blockwise full size N={N} K={K}")
    c = workloads.blockwise_case(q, N, K, B, rb, seed=1)
    y = run(c)
    rows = np.sort(np.random.default_rng(0).choice(N, 512, replace=False))
    rows[-1] = N - 1
    y_ref, a_ref = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb,
                                                  rows=rows)
    check(y[:, rows], y_ref, a_ref, f"{N}x{K} sampled")


def test_blockwise_error_codes():
    c = workloads.blockwise_case(2, 64, 256, 1, 8, seed=1)
    packed = sa.pack_weights(dev(c["signs"]))
    y = torch.empty((1, 64), dtype=torch.float32, device="cuda")
    with pytest.raises(sa.SaError):
        sa.sa_shiftadd_gemm_blockwise(dev(c["x"]), packed, dev(c["blk_exps"]), 9, 64, 256, 8, 1,
                                      y)
    with pytest.raises(sa.SaError):
        sa.sa_shiftadd_gemm_blockwise(dev(c["x"]), packed, dev(c["blk_exps"]), 2, 64, 256, 0, 1,
                                      y)


# Batch >= 2 runs the batch kernel (plan path 5): 16, 32 or 64 rows per
# workgroup (KW = 1, 2, 4 key words per lane) and four batch rows per table.
# When row_block is a multiple of the workgroup's rows the block exponents
# come in by scalar loads ("uniform"), else per lane.
BATCH_CASES = [
    # (q, N, K, B, row_block, label)
    (3, 1000, 1024, 8, 125, "KW=1, two quads, per lane"),
    (3, 4096, 1024, 8, 512, "KW=2, uniform"),
    (4, 4096, 512, 16, 512, "four planes (KW capped at 2), uniform"),
    (3, 4096, 2048, 16, 512, "KW=4, uniform"),
    (2, 4096, 1024, 16, 100, "KW=4, per lane"),
    (3, 4000, 1024, 16, 512, "uniform, ragged last tile"),
    (3, 4000, 1024, 16, 1000, "KW=4, q=3, per lane"),
    (8, 2048, 512, 16, 256, "KW=2, eight planes, uniform"),
    (2, 130, 384, 5, 17, "ragged quad and rows, 17-row blocks"),
    (1, 77, 4224, 6, 1, "a factor per row, ragged last piece"),
    (5, 300, 2048, 13, 40, "five planes, two pieces, ragged quad"),
]


@pytest.mark.parametrize("q,N,K,B,rb,label", BATCH_CASES, ids=[c[-1] for c in BATCH_CASES])
def test_blockwise_batch_parity(q, N, K, B, rb, label):
    plan = sa.sa_plan_gemm_blockwise(q, N, K, rb, B)
    assert plan["path"] == 5
    assert ("uniform" in label) == (rb % plan["rows_per_wg"] == 0)
    say(f"blockwise batch q={q} N={N} K={K} B={B} row_block={rb} "
        f"rows/wg={plan['rows_per_wg']}: {label}")
    c = workloads.blockwise_case(q, N, K, B, rb, seed=q + N + K + B + rb)
    y = run(c)
    y_ref, a_ref = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb)
    check(y, y_ref, a_ref, label)


def test_blockwise_batch_rows_agree_with_batch_one():
    """Each batch row of the batch kernel against the row kernel on that row
    alone (another kernel), within the bar of both against the oracle."""
    q, N, K, B, rb = 3, 1024, 2048, 8, 128
    c = workloads.blockwise_case(q, N, K, B, rb, seed=5)
    y = run(c)
    y_ref, a_ref = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb)
    check(y, y_ref, a_ref, "batch 8")
    for b in (0, 5, 7):
        one = dict(c, B=1, x=c["x"][b:b + 1])
        y1 = run(one)
        check(y1, y_ref[b:b + 1], a_ref[b:b + 1], f"batch row {b} alone")


@pytest.mark.parametrize("N,K", [(4096, 4096), (11008, 4096)])
def test_blockwise_batch_full_size_sampled(N, K):
    """LLaMA-2-7B projection shapes, q = 3, batch 16, row_block = N / 8; 256
    sampled rows."""
    q, B, rb = 3, 16, N // 8
    say(f"blockwise batch full size N={N} K={K} B={B}")
    c = workloads.blockwise_case(q, N, K, B, rb, seed=2)
    y = run(c)
    rows = np.sort(np.random.default_rng(1).choice(N, 256, replace=False))
    rows[-1] = N - 1
    y_ref, a_ref = oracle.shiftadd_gemm_blockwise(c["x"], c["signs"], c["blk_exps"], rb,
                                                  rows=rows)
    check(y[:, rows], y_ref, a_ref, f"{N}x{K} batch {B} sampled")
