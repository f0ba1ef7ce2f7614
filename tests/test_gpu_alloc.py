"""GPU parity of the criterion of Eq. 3 (sa_gram_f16, sa_inverse_cholesky_diag,
sa_importance_criterion) against the CPU oracle (oracle/alloc.py).

Bars (fixed here):
* Gram matrix: |H - X X^T| <= 2 T 2^-24 (|X| |X|^T) elementwise (fp16 products
  are exact in fp32; only the fp32 accumulation rounds).
* d = diag(cholesky(H^-1)) from the same fp32 H: relative 1e-9 (two fp64
  factorizations of a matrix damped to a condition number of a few thousand
  at most).
* C from the same d: relative 1e-12 (fp64 sums in different orders).
* End to end from X: relative 1e-4 (the fp32 Gram matrix against fp64).
"""
import sys

import numpy as np
import pytest

from oracle import alloc
import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - CPU-only environment
    pytest.skip("no GPU", allow_module_level=True)
sa = pytest.importorskip("paper_2406_05981_amd.shiftadd")


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def calib(K, T, seed, outliers=0.01):
    """fp16 calibration activations [K][T]: N(0,1) with outlier channels x20."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((K, T))
    n_out = int(round(outliers * K))
    if n_out:
        x[rng.choice(K, n_out, replace=False)] *= 20.0
    return x.astype(np.float16)


def gpu_gram(x16):
    K, T = x16.shape
    H = torch.empty((K, K), dtype=torch.float32, device="cuda")
    sa.sa_gram_f16(torch.from_numpy(x16).cuda(), K, T, H)
    torch.cuda.synchronize()
    return H


def gpu_d(H, damp):
    K = H.shape[0]
    d = torch.empty(K, dtype=torch.float64, device="cuda")
    ws = torch.empty(sa.lib.sa_inverse_cholesky_workspace(K), dtype=torch.uint8, device="cuda")
    sa.sa_inverse_cholesky_diag(H, K, damp, d, ws)
    torch.cuda.synchronize()
    return d.cpu().numpy()


@pytest.mark.parametrize("K,T", [(128, 32), (128, 96), (256, 512), (512, 2048), (1024, 160),
                                 # the large-shape path (K >= 1024, T >= 16384): whole super-panels,
                                 # a half-empty last super-panel (K % 256 == 128), T an odd multiple of 32
                                 (1024, 16384), (1152, 16416)])
def test_gram(K, T):
    say(f"gram K={K} T={T}")
    x = calib(K, T, seed=K + T)
    H = gpu_gram(x).cpu().numpy().astype(np.float64)
    x64 = x.astype(np.float64)
    ref = x64 @ x64.T
    bound = 2 * T * 2.0 ** -24 * (np.abs(x64) @ np.abs(x64).T)
    assert (np.abs(H - ref) <= bound).all()
    assert np.array_equal(H, H.T)


@pytest.mark.parametrize("K,T", [(128, 96), (1152, 16416)])
def test_gram_repeatable(K, T):
    """Two calls give the same bits (the large-shape path adds exactly two
    partials onto zero per entry, and sums the column pieces of the leftover
    quadrants in a fixed order)."""
    say(f"gram repeatable K={K} T={T}")
    x = torch.from_numpy(calib(K, T, seed=7)).cuda()
    H1 = torch.empty((K, K), dtype=torch.float32, device="cuda")
    H2 = torch.full((K, K), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_gram_f16(x, K, T, H1)
    sa.sa_gram_f16(x, K, T, H2)
    torch.cuda.synchronize()
    assert torch.equal(H1, H2)


@pytest.mark.parametrize("K,T,damp", [(64, 256, 0.01), (200, 512, 0.01), (384, 256, 0.05),
                                      (1000, 2048, 0.01), (130, 1024, 0.0),
                                      # last diagonal block of 1, 63 and 1 rows; whole panels only
                                      (65, 256, 0.01), (127, 512, 0.01), (129, 512, 0.01),
                                      (256, 1024, 0.01),
                                      # one partial diagonal block only
                                      (1, 32, 0.01), (2, 32, 0.0), (63, 256, 0.01)])
def test_inverse_cholesky_diag(K, T, damp):
    """Including K not a multiple of the 64-column panel, and no damping on a
    full-rank calibration set."""
    say(f"inverse cholesky diag K={K} T={T} damp={damp}")
    x = calib(K, T, seed=K)
    x64 = x.astype(np.float64)
    H32 = (x64 @ x64.T).astype(np.float32)      # any symmetric fp32 input
    d = gpu_d(torch.from_numpy(H32).cuda(), damp)
    ref = alloc.cholesky_diag_of_inverse(alloc.damped(H32.astype(np.float64), damp))
    assert np.all(np.isfinite(d))
    assert np.allclose(d, ref, rtol=1e-9, atol=0)


@pytest.mark.parametrize("K,m", [(300, 100), (200, 199), (130, 0)])
def test_inverse_cholesky_not_positive_definite(K, m):
    """The documented behaviour for a matrix that is not positive definite:
    channel m made to fail (its pivot, taken after the later channels in the
    reversed order, is negative).  d[k] for k > m depends only on the later
    channels and matches the oracle on that trailing block; d[0..m] are NaN."""
    say(f"not positive definite K={K} m={m}")
    x = calib(K, 4 * K, seed=K + m)
    x64 = x.astype(np.float64)
    H = x64 @ x64.T
    H[m, m] = -1000.0 * abs(H[m, m])
    H32 = H.astype(np.float32)
    d = gpu_d(torch.from_numpy(H32).cuda(), 0.0)
    assert np.all(np.isnan(d[:m + 1]))
    if m + 1 < K:
        ref = alloc.cholesky_diag_of_inverse(alloc.damped(H32[m + 1:, m + 1:].astype(np.float64), 0.0))
        assert np.all(np.isfinite(d[m + 1:]))
        assert np.allclose(d[m + 1:], ref, rtol=1e-9, atol=0)


def test_criterion_from_d():
    N, K = 300, 256
    w = workloads.fp_weights(N, K, seed=3)
    rng = np.random.default_rng(4)
    d = rng.uniform(0.01, 1.0, K)
    out = torch.empty(3, dtype=torch.float64, device="cuda")
    ws = torch.empty(sa.lib.sa_importance_workspace(), dtype=torch.uint8, device="cuda")
    sa.sa_importance_criterion(torch.from_numpy(w).cuda(), N, K, torch.from_numpy(d).cuda(), out, ws)
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    IS = w.astype(np.float64) / d[None, :]
    assert o[0] == pytest.approx(np.linalg.norm(IS) * IS.std() ** 2, rel=1e-12)
    assert o[1] == pytest.approx(np.linalg.norm(IS), rel=1e-12)
    assert o[2] == pytest.approx(IS.std(), rel=1e-12)


@pytest.mark.parametrize("N,K,T", [(128, 128, 1024), (1024, 1024, 4096), (4096, 2048, 8192),
                                   (512, 1024, 16384)])
def test_criterion_end_to_end(N, K, T):
    """Eq. 3 for one layer from its weights and fp16 calibration activations;
    the largest case is a 2048-channel layer with 8192 calibration tokens."""
    say(f"criterion end to end N={N} K={K} T={T}")
    w = workloads.fp_weights(N, K, seed=K)
    x = calib(K, T, seed=T)
    C, fro, std, d = sa.bit_criterion(torch.from_numpy(w).cuda(), torch.from_numpy(x).cuda(), 0.01)
    ref = alloc.criterion(w, x.astype(np.float64), 0.01)
    say(f"  C = {C:.6e}, oracle {ref:.6e}")
    assert C == pytest.approx(ref, rel=1e-4)


def test_criterion_full_size():
    """The criterion at the size `bench.py --criterion` times: N = K = 4096 and
    262144 calibration tokens (the large-shape Gram path, 64 Cholesky panels),
    activations drawn as there.  Sampled Gram entries (off-diagonal regions,
    diagonal regions and their leftover quadrants) against exact fp64 dot
    products within the Gram bar, the whole matrix symmetric; d for all 4096
    channels against the oracle from the same fp32 H (relative 1e-9); C, ||IS||
    and STD(IS) against fp64 statistics of the same d (relative 1e-12)."""
    N = K = 4096
    T = 262144
    say(f"criterion full size N={N} K={K} T={T}: drawing activations")
    rng = np.random.default_rng(0)
    x16 = np.empty((K, T), np.float16)
    out_rows = set(rng.choice(K, K // 100, replace=False).tolist())
    for r0 in range(0, K, 256):   # row blocks: 4 GB of fp32 draws at once otherwise
        blk = rng.standard_normal((256, T), dtype=np.float32)
        for r in range(256):
            if r0 + r in out_rows:
                blk[r] *= 20.0
        x16[r0:r0 + 256] = blk.astype(np.float16)
    say("  gram")
    H = gpu_gram(x16)
    Hn = H.cpu().numpy()
    assert np.array_equal(Hn, Hn.T)
    pairs = [(int(i), int(j)) for i, j in zip(rng.integers(0, K, 48), rng.integers(0, K, 48))]
    for a in rng.integers(0, K // 256, 8):        # inside diagonal 256 x 256 regions
        base = 256 * int(a)
        pairs += [(base + int(rng.integers(192, 256)), base + int(rng.integers(128, 256))),
                  (base + int(rng.integers(0, 256)), base + int(rng.integers(0, 256)))]
    for i, j in pairs:
        xi, xj = x16[i].astype(np.float64), x16[j].astype(np.float64)
        ref = xi @ xj
        bound = 2 * T * 2.0 ** -24 * (np.abs(xi) @ np.abs(xj))
        assert abs(float(Hn[i, j]) - ref) <= bound, (i, j, float(Hn[i, j]), ref)
    del x16
    say("  inverse cholesky diag")
    d = gpu_d(H, 0.01)
    ref_d = alloc.cholesky_diag_of_inverse(alloc.damped(Hn.astype(np.float64), 0.01))
    assert np.all(np.isfinite(d))
    assert np.allclose(d, ref_d, rtol=1e-9, atol=0)
    say("  importance")
    w = workloads.fp_weights(N, K, seed=1)
    out = torch.empty(3, dtype=torch.float64, device="cuda")
    ws = torch.empty(sa.lib.sa_importance_workspace(), dtype=torch.uint8, device="cuda")
    sa.sa_importance_criterion(torch.from_numpy(w).cuda(), N, K, torch.from_numpy(d).cuda(), out, ws)
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    IS = w.astype(np.float64) / d[None, :]
    assert o[0] == pytest.approx(np.linalg.norm(IS) * IS.std() ** 2, rel=1e-12)
    assert o[1] == pytest.approx(np.linalg.norm(IS), rel=1e-12)
    assert o[2] == pytest.approx(IS.std(), rel=1e-12)


def test_allocation_pipeline():
    """Criteria of a few synthetic layers -> per-bit fits against measured
    quantization errors (the GPU quantizer at 2, 3, 4 bits, weighted by the
    calibration Gram matrix) -> Eq. 4.  The result meets the budget, and the
    layer with the largest criterion gets at least as many bits as the one
    with the smallest."""
    K, T, G = 256, 1024, 128
    x = calib(K, T, seed=5)
    xg = torch.from_numpy(x).cuda()
    H = gpu_gram(x).cpu().numpy().astype(np.float64)
    crit, errs = [], []
    for i, scale in enumerate([0.005, 0.01, 0.02, 0.04, 0.08, 0.16]):
        w = workloads.fp_weights(128, K, seed=i, scale=scale)
        C, _, _, _ = sa.bit_criterion(torch.from_numpy(w).cuda(), xg, 0.01)
        crit.append(C)
        e = []
        for q in (2, 3, 4):
            s, ex = sa.quantize_bcq(torch.from_numpy(w).cuda(), q, G, 2)
            wq = (np.ldexp(1.0, np.repeat(ex.cpu().numpy().astype(np.int64), G, axis=2))
                  * s.cpu().numpy()).sum(0)
            dlt = wq - w
            e.append(float(np.einsum("nk,kl,nl->", dlt, H, dlt)))
        errs.append(e)
    est = sa.sa_fit_per_bit(np.array(crit), np.array(errs), 1)
    widths, obj = sa.sa_allocate_bits(est, [2, 3, 4], 3.0)
    ref_w, _ = alloc.allocate(est, [2, 3, 4], 3.0)
    assert widths.tolist() == ref_w.tolist()
    assert widths.sum() <= 3 * len(widths)
    assert widths[int(np.argmax(crit))] >= widths[int(np.argmin(crit))]
