"""GPU parity of the layer with additive power-of-two factors
(sa_shiftadd_gemm_terms, Eq. 2 with T terms) against the CPU oracle
(oracle.shiftadd_gemm_terms).

Bar (fixed here): max |y - y_ref| / sum|terms| <= 2e-3 per output, with the
1e-5 alarm of the fp32 tables (each term is an exact shift of the fp32 group
sum)."""
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
    q, N, K, G, B, T = c["q"], c["N"], c["K"], c["G"], c["B"], c["T"]
    y = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm_terms(dev(c["x"]), sa.pack_weights(dev(c["signs"])), dev(c["exps"]),
                              dev(c["term_signs"]), q, N, K, G, T, B, y)
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
    # (q, N, K, G, B, T, label)
    (3, 768, 768, 128, 1, 2, "two terms, one piece"),
    (2, 130, 384, 384, 1, 3, "G = K, ragged rows, three terms"),
    (1, 33, 128, 128, 3, 4, "four terms, batch 3"),
    (4, 4100, 1024, 256, 2, 2, "G = 256, several row groups per workgroup"),
    (3, 64, 8192, 128, 1, 3, "two pieces"),
    (8, 17, 256, 128, 1, 2, "eight planes"),
    (3, 300, 4224, 128, 2, 4, "ragged last piece"),
    (3, 1000, 8320, 128, 1, 2, "16 waves, three pieces, one-block last piece"),
    (2, 4096, 8192, 256, 1, 3, "16 waves, 256 workgroups, G = 256"),
    (3, 8000, 8320, 128, 1, 2, "16 waves, two row groups per workgroup"),
]


@pytest.mark.parametrize("q,N,K,G,B,T,label", CASES, ids=[c[-1] for c in CASES])
def test_terms_parity(q, N, K, G, B, T, label):
    say(f"terms q={q} N={N} K={K} G={G} B={B} T={T}: {label}")
    c = workloads.terms_case(q, N, K, G, B, T, seed=q + N + K + B + T)
    y = run(c)
    y_ref, a_ref = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], G)
    check(y, y_ref, a_ref, label)


def test_one_term_matches_row_wise_kernel():
    q, N, K, G, B = 3, 512, 2048, 128, 1
    c = workloads.terms_case(q, N, K, G, B, 1, seed=11)
    y = run(c)
    yr = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm(dev(c["x"]), sa.pack_weights(dev(c["signs"])), dev(c["exps"][..., 0]), q,
                        N, K, G, B, yr)
    torch.cuda.synchronize()
    assert np.array_equal(y, yr.cpu().numpy().astype(np.float64))  # same arithmetic


def test_terms_full_size_sampled():
    q, N, K, G, B, T = 3, 4096, 4096, 128, 1, 2
    say("terms full size 4096x4096 T=2")
    c = workloads.terms_case(q, N, K, G, B, T, seed=1)
    y = run(c)
    rows = np.sort(np.random.default_rng(0).choice(N, 512, replace=False))
    y_ref, a_ref = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], G,
                                              rows=rows)
    check(y[:, rows], y_ref, a_ref, "4096x4096 sampled")


# Batch >= 2 runs the batch kernel: 16, 32 or 64 rows per workgroup and four
# batch rows per table.
BATCH_CASES = [
    # (q, N, K, G, B, T, label)
    (3, 1000, 1024, 128, 8, 2, "KW=1, two quads"),
    (3, 4096, 1024, 256, 8, 3, "KW=2, G = 256, three terms"),
    (4, 4096, 512, 128, 16, 4, "KW=4, four terms"),
    (8, 2048, 512, 512, 16, 2, "KW=2, eight planes, G = K"),
    (2, 130, 384, 384, 5, 3, "ragged quad and rows"),
    (1, 77, 4224, 128, 6, 4, "ragged last piece"),
    (5, 300, 2048, 1024, 13, 2, "five planes, two pieces, ragged quad"),
    # exponents and term signs preloaded per lane (G = 128, K % 1024 == 0)
    (3, 1000, 4096, 128, 8, 2, "preloaded, 8 bytes"),
    (2, 500, 8192, 128, 5, 2, "preloaded, 16 bytes"),
    (3, 300, 4096, 128, 6, 4, "preloaded, 16 bytes, four terms"),
    (1, 64, 2048, 128, 4, 4, "preloaded, 8 bytes, two pieces"),
    (3, 200, 4096, 128, 4, 1, "preloaded, one term"),
    (4, 300, 4096, 128, 8, 2, "four planes: per-piece loads"),
    (3, 300, 4096, 128, 8, 3, "three terms: per-piece loads"),
]


@pytest.mark.parametrize("q,N,K,G,B,T,label", BATCH_CASES, ids=[c[-1] for c in BATCH_CASES])
def test_terms_batch_parity(q, N, K, G, B, T, label):
    assert sa.sa_plan_gemm(q, N, K, G, B)["path"] == 2
    say(f"terms batch q={q} N={N} K={K} G={G} B={B} T={T}: {label}")
    c = workloads.terms_case(q, N, K, G, B, T, seed=q + N + K + B + T)
    y = run(c)
    y_ref, a_ref = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], G)
    check(y, y_ref, a_ref, label)


def test_one_term_batch_matches_row_wise_batch_kernel():
    q, N, K, G, B = 3, 2048, 2048, 128, 8
    c = workloads.terms_case(q, N, K, G, B, 1, seed=12)
    assert (c["term_signs"] != 0).all()
    y = run(c)
    yr = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm(dev(c["x"]), sa.pack_weights(dev(c["signs"])), dev(c["exps"][..., 0]), q,
                        N, K, G, B, yr)
    torch.cuda.synchronize()
    assert np.array_equal(y, yr.cpu().numpy().astype(np.float64))  # same arithmetic


def test_one_term_batch_matches_row_wise_batch_kernel_preloaded():
    """K = 4096: the additive kernel preloads its exponents and term signs,
    the row-wise kernel loads them per piece; still the same arithmetic."""
    q, N, K, G, B = 3, 1024, 4096, 128, 8
    c = workloads.terms_case(q, N, K, G, B, 1, seed=13)
    assert (c["term_signs"] != 0).all()
    y = run(c)
    yr = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm(dev(c["x"]), sa.pack_weights(dev(c["signs"])), dev(c["exps"][..., 0]), q,
                        N, K, G, B, yr)
    torch.cuda.synchronize()
    assert np.array_equal(y, yr.cpu().numpy().astype(np.float64))


@pytest.mark.parametrize("shift", [4, 8])
def test_terms_batch_misaligned(shift):
    """Exponents and term signs at addresses not aligned to the 16-byte preload
    take the per-piece loads: the same arithmetic, so bit-identical output."""
    q, N, K, G, B, T = 3, 700, 8192, 128, 6, 2
    say(f"terms batch misaligned by {shift}")
    c = workloads.terms_case(q, N, K, G, B, T, seed=31)
    y_al = run(c)

    def shifted(a):
        flat = torch.from_numpy(np.ascontiguousarray(a).reshape(-1)).cuda()
        buf = torch.zeros(flat.numel() + 32, dtype=torch.int8, device="cuda")
        view = buf[shift:shift + flat.numel()]
        view.copy_(flat)
        return view.view(a.shape)

    y = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm_terms(dev(c["x"]), sa.pack_weights(dev(c["signs"])), shifted(c["exps"]),
                              shifted(c["term_signs"]), q, N, K, G, T, B, y)
    torch.cuda.synchronize()
    y_mis = y.cpu().numpy().astype(np.float64)
    assert np.array_equal(y_al, y_mis)
    y_ref, a_ref = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], G)
    check(y_mis, y_ref, a_ref, "misaligned exponents and term signs")


def test_terms_batch_full_size_sampled():
    q, N, K, G, B, T = 3, 4096, 4096, 128, 16, 2
    say("terms batch full size 4096x4096 B=16 T=2")
    c = workloads.terms_case(q, N, K, G, B, T, seed=2)
    y = run(c)
    rows = np.sort(np.random.default_rng(1).choice(N, 256, replace=False))
    rows[-1] = N - 1
    y_ref, a_ref = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], G,
                                              rows=rows)
    check(y[:, rows], y_ref, a_ref, "4096x4096 batch 16 sampled")


@pytest.mark.parametrize("B", [1, 2, 8])
@pytest.mark.parametrize("K", [1024, 4096])
def test_sign_zero_terms_ignore_their_exponent(B, K):
    """A term sign of 0 means no term, whatever its exponent byte holds: with
    every sign-0 term carrying exponent 127 (2^127 times a group sum overflows
    fp32) the row kernel (batch 1) and the batch kernel (batch >= 2, per-piece
    and preloaded exponents) still match the oracle, which skips such terms."""
    q, N, G, T = 3, 300, 128, 3
    say(f"sign-0 terms with exponent 127: K={K} B={B}")
    c = workloads.terms_case(q, N, K, G, B, T, seed=41 + B + K)
    zero = c["term_signs"] == 0
    assert zero.any()
    c["exps"][zero] = 127
    y = run(c)
    y_ref, a_ref = oracle.shiftadd_gemm_terms(c["x"], c["signs"], c["exps"], c["term_signs"], G)
    check(y, y_ref, a_ref, f"sign-0 terms, exponent 127, batch {B}")
