"""GPU parity of the offline reparameterization (sa_quantize_bcq) against the
CPU oracle (oracle/bcq.py).

Bar: the sign planes and the int8 exponents are integers decided by fp64
arithmetic on both sides, so they must be bit-identical.  The two sides keep
every operation of the algorithm in the same order except the order of two
segment sums (sum|r| in the greedy step and B^T w in the least-squares step),
which may round differently in the last bit.  A segment whose output differs is
accepted only when the oracle's own path through it passes within 1e-9
(relative) of a decision boundary -- a sign decision on a residual, the
power-of-two rounding boundary, or a tie between the two nearest code values --
so that a last-bit difference can flip it.  Every other segment must match
exactly.
"""
import sys

import numpy as np
import pytest

import workloads
from oracle import bcq

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - CPU-only environment
    pytest.skip("no GPU", allow_module_level=True)
sa = pytest.importorskip("paper_2406_05981_amd.shiftadd")

MARGIN = 1e-9


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def gpu_quantize(w, q, G, T):
    signs, exps = sa.quantize_bcq(torch.from_numpy(np.ascontiguousarray(w)).cuda(), q, G, T)
    torch.cuda.synchronize()
    return signs.cpu().numpy(), exps.cpu().numpy()


def min_margin(seg, q, T):
    """Smallest relative distance of the oracle's decisions on one segment from
    a boundary where a last-bit change of a sum could flip them."""
    w = seg[None, :].astype(np.float64)
    scale = max(float(np.abs(w).max()), 1e-300)
    margins = []
    # greedy sign decisions on the residuals
    r = w.copy()
    B, A = bcq.greedy(w, q)
    for i in range(q):
        margins.append(np.abs(r).min() / scale)
        r = r - A[:, i:i + 1] * B[:, i]

    def pot_margin(alpha):
        mag = np.abs(alpha[alpha != 0])
        if mag.size == 0:
            return np.inf
        l2 = np.log2(mag)
        return float(np.abs(l2 - np.floor(l2) - 0.5).min())

    def bs_margin(pa):
        vals = bcq.code_values(pa)
        dist = np.sort(np.abs(w[:, :, None] - vals[:, None, :]), axis=2)
        gaps = dist[:, :, 1] - dist[:, :, 0]
        gaps = gaps[gaps > 0]  # exact ties are decided identically
        return float(gaps.min() / scale) if gaps.size else np.inf

    if T == 0:
        margins.append(pot_margin(A))
    for _ in range(T):
        A = bcq.least_squares(B, w)
        margins.append(pot_margin(A))
        pa = bcq.pot_values(A)
        margins.append(bs_margin(pa))
        B = bcq.binary_search(pa, w)
    return min(margins)


def check_parity(w, q, G, T, label):
    say(f"[bcq] {label}: N={w.shape[0]} K={w.shape[1]} q={q} G={G} T={T}")
    s_gpu, e_gpu = gpu_quantize(w, q, G, T)
    s_ref, e_ref = bcq.quantize(w, q, G, T)
    assert s_gpu.shape == s_ref.shape and e_gpu.shape == e_ref.shape
    assert set(np.unique(s_gpu)) <= {-1, 1}
    N, K = w.shape
    NG = K // G
    bad_s = (s_gpu != s_ref).reshape(q, N, NG, G).any(axis=(0, 3))
    bad_e = (e_gpu != e_ref).any(axis=0)
    bad = np.argwhere(bad_s | bad_e)
    for n, g in bad:
        m = min_margin(w[n, g * G:(g + 1) * G], q, T)
        assert m < MARGIN, f"{label}: segment (row {n}, group {g}) differs, oracle margin {m:.3e}"
    if len(bad):
        say(f"[bcq] {label}: {len(bad)} of {N * NG} segments differ, each at a near-tie")
    return s_gpu, e_gpu


SHAPES = [
    # (q, N, K, G, T, label)
    (1, 64, 256, 128, 0, "q=1 greedy only"),
    (1, 37, 384, 128, 3, "q=1 (closed form, LS leaves it fixed)"),
    (2, 100, 384, 128, 3, "q=2"),
    (3, 130, 512, 128, 2, "q=3, ragged row count"),
    (3, 64, 1024, 128, 0, "q=3 greedy + PoT only"),
    (4, 70, 1024, 256, 2, "q=4, G=256 (4 elements per lane)"),
    (5, 17, 96, 8, 4, "q=5 > log2(G): dependent planes, G=8"),
    (6, 9, 200, 40, 3, "q=6, G=40 (ragged lanes)"),
    (7, 12, 192, 192, 1, "q=7, G=K=192"),
    (8, 33, 512, 64, 2, "q=8, 256-entry code table"),
    (3, 5, 4096, 4096, 2, "q=3, G=K=4096 (wave per segment, 64 elements per lane)"),
    (2, 20, 1056, 264, 2, "q=2, G=264 (wave per segment, ragged lanes)"),
    (4, 6, 2048, 512, 3, "q=4, G=512 (wave per segment)"),
    (6, 9, 1024, 512, 2, "q=6, G=512 (wave per segment, table in LDS)"),
]


@pytest.mark.parametrize("q,N,K,G,T,label", SHAPES, ids=[s[-1] for s in SHAPES])
def test_quantize_parity(q, N, K, G, T, label):
    w = workloads.fp_weights(N, K, seed=q * 7 + T)
    check_parity(w, q, G, T, label)


@pytest.mark.parametrize("G", [64, 512])
def test_quantize_edge_values(G):
    """Zero segments, constant segments, exactly representable ties, fp32
    extremes (power-of-two exponents clamped to [-128, 127]) and subnormals,
    through both kernels (16 lanes per segment, and one wave per segment)."""
    q, T = 3, 2
    rows = []
    rows.append(np.zeros(256))
    rows.append(np.full(256, 0.375))
    rows.append(np.tile([3, 1, -1, -3, 3, 1, -1, -2], 32) * 0.5)   # hand segment with a tie
    rows.append(np.concatenate([np.full(128, 3e38), np.full(128, -3e38)]))
    rows.append(np.full(256, 1e-44))                               # fp32 subnormals
    rows.append(np.concatenate([np.full(64, 1e-30), np.full(64, -2.0 ** -126),
                                np.linspace(-1, 1, 128)]))
    rng = np.random.default_rng(5)
    rows.append(rng.choice([-0.25, 0.25, 0.75, -0.75], size=256))   # 2-plane PoT values
    w = np.tile(np.stack(rows), (1, 2)).astype(np.float32)
    for T_ in (0, T):
        s, e = check_parity(w, q, G, T_, f"edge values G={G} T={T_}")
    # the fp32 extremes clamp at the top of the exponent range
    assert e[:, 3].max() == 127
    # zero segments: no scale, all exponents at the bottom of the range
    assert (e[:, 0] == -128).all()


def test_quantize_recovers_formatted_weights():
    """Weights that already have the format (powers of two times sign planes)
    come back exactly after one cycle for q <= 2."""
    for q in (1, 2):
        c = workloads.random_case(q, 48, 512, 128, 1, seed=11, exp_range=(-6, -3))
        scale = np.ldexp(1.0, np.repeat(c["exps"].astype(np.int64), 128, axis=2))
        w = (scale * c["signs"]).sum(axis=0).astype(np.float32)
        s, e = check_parity(w, q, 128, 1, f"formatted q={q}")
        assert np.array_equal(bcq.reconstruct(s, e, 128), w.astype(np.float64))


def test_quantize_two_calls_and_error_codes():
    w = torch.from_numpy(workloads.fp_weights(16, 256, seed=3)).cuda()
    s1, e1 = sa.quantize_bcq(w, 3, 128, 2)
    s2, e2 = sa.quantize_bcq(w, 3, 128, 2)
    torch.cuda.synchronize()
    assert torch.equal(s1, s2) and torch.equal(e1, e2)  # deterministic
    with pytest.raises(sa.SaError):
        sa.quantize_bcq(w, 3, 96, 2)
    with pytest.raises(sa.SaError):
        sa.quantize_bcq(w, 9, 128, 2)
    with pytest.raises(sa.SaError):
        sa.quantize_bcq(w, 3, 128, sa.SA_MAX_CYCLES + 1)


def test_quantize_full_layer_sampled():
    """A LLaMA-2-7B attention projection (4096 x 4096, q = 3, G = 128, T = 2)
    in the launch configuration the benchmark times; 1024 sampled segments are
    compared with the oracle, and the relative error of the whole layer must
    agree with the oracle's on the sample (outliers make it larger than on
    Gaussian weights alone)."""
    N = K = 4096
    q, G, T = 3, 128, 2
    w = workloads.fp_weights(N, K, seed=1)
    say(f"[bcq] full layer N={N} K={K} q={q} G={G} T={T}")
    s, e = gpu_quantize(w, q, G, T)
    assert set(np.unique(s)) <= {-1, 1}
    assert e.min() >= -128 and e.max() <= 127
    rng = np.random.default_rng(0)
    NG = K // G
    picks = rng.choice(N * NG, size=1024, replace=False)
    segs = np.stack([w[p // NG, (p % NG) * G:(p % NG + 1) * G] for p in picks])
    s_ref, e_ref = bcq.quantize(segs, q, G, T)   # segments as rows of one group
    bad = 0
    for j, p in enumerate(picks):
        n, g = divmod(int(p), NG)
        same = (np.array_equal(s[:, n, g * G:(g + 1) * G], s_ref[:, j, :])
                and np.array_equal(e[:, n, g], e_ref[:, j, 0]))
        if not same:
            bad += 1
            m = min_margin(segs[j], q, T)
            assert m < MARGIN, f"segment (row {n}, group {g}) differs, oracle margin {m:.3e}"
    say(f"[bcq] full layer: {bad} of {len(picks)} sampled segments at near-ties differ")
    wq = bcq.reconstruct(s, e, G)
    rel = np.linalg.norm(wq - w) / np.linalg.norm(w)
    seg_q = bcq.reconstruct(s_ref, e_ref, G)
    rel_ref = np.linalg.norm(seg_q - segs) / np.linalg.norm(segs)
    say(f"[bcq] full layer relative error {rel:.4f} (oracle on the sample {rel_ref:.4f})")
    assert rel < 0.5 and abs(rel - rel_ref) < 0.1 * rel_ref


def test_quantize_then_layer():
    """The front-end feeds the layer: quantize on the GPU, pack, run the layer;
    the result agrees with the oracle's layer on the same planes and with the
    dense product of the reconstructed weights."""
    import oracle

    N, K, q, G, T = 512, 1024, 3, 128, 2
    w = workloads.fp_weights(N, K, seed=21)
    s_dev, e_dev = sa.quantize_bcq(torch.from_numpy(w).cuda(), q, G, T)
    packed = sa.pack_weights(s_dev)
    x = (np.random.default_rng(1).standard_normal((2, K))).astype(np.float16)
    y = sa.shiftadd_gemm(torch.from_numpy(x).cuda(), packed, e_dev, q, N, K, G)
    torch.cuda.synchronize()
    y = y.cpu().numpy().astype(np.float64)
    s, e = s_dev.cpu().numpy(), e_dev.cpu().numpy()
    y_ref, a_ref = oracle.shiftadd_gemm(x, s, e, G)
    assert (np.abs(y - y_ref) / a_ref).max() <= 2e-3
    y_dense = x.astype(np.float64) @ bcq.reconstruct(s, e, G).T
    assert np.abs(y_ref - y_dense).max() <= 1e-12 * a_ref.max()


# ------------------------------------------------------------ additive PoT scales

def gpu_quantize_terms(w, q, G, T, terms):
    s, e, t = sa.quantize_bcq_terms(torch.from_numpy(np.ascontiguousarray(w)).cuda(), q, G, T,
                                    terms)
    torch.cuda.synchronize()
    return s.cpu().numpy(), e.cpu().numpy(), t.cpu().numpy()


TERM_SHAPES = [
    # (q, N, K, G, T, terms, label)
    (3, 130, 512, 128, 2, 1, "one term: the single-term format"),
    (3, 130, 512, 128, 2, 2, "two terms"),
    (2, 64, 1024, 256, 3, 3, "three terms, G = 256"),
    (4, 40, 384, 64, 0, 4, "four terms, greedy scales only"),
    (6, 9, 1024, 512, 2, 2, "q = 6, wave per segment"),
    (3, 5, 4096, 4096, 1, 3, "G = K"),
]


@pytest.mark.parametrize("q,N,K,G,T,terms,label", TERM_SHAPES, ids=[c[-1] for c in TERM_SHAPES])
def test_quantize_terms_parity(q, N, K, G, T, terms, label):
    say(f"[bcq terms] {label}: N={N} K={K} q={q} G={G} T={T} terms={terms}")
    w = workloads.fp_weights(N, K, seed=q * 13 + terms)
    s, e, t = gpu_quantize_terms(w, q, G, T, terms)
    s_ref, e_ref, t_ref = bcq.quantize_terms(w, q, G, T, terms)
    NG = K // G
    bad = ((s != s_ref).reshape(q, N, NG, G).any(axis=(0, 3)) |
           (e != e_ref).any(axis=(0, 3)) | (t != t_ref).any(axis=(0, 3)))
    assert not bad.any(), f"{label}: {int(bad.sum())} segments differ"
    if terms == 1:
        s1, e1 = gpu_quantize(w, q, G, T)
        assert np.array_equal(s, s1) and np.array_equal(e[..., 0], e1)


def test_quantize_terms_then_layer():
    """Additive scales end to end: quantize with two terms, pack, run the
    additive layer; agrees with the oracle's additive layer on the same planes
    and with the dense product of the reconstructed weights."""
    import oracle

    N, K, q, G, T, terms = 512, 1024, 3, 128, 2, 2
    w = workloads.fp_weights(N, K, seed=22)
    s_d, e_d, t_d = sa.quantize_bcq_terms(torch.from_numpy(w).cuda(), q, G, T, terms)
    x = np.random.default_rng(2).standard_normal((2, K)).astype(np.float16)
    y = torch.empty((2, N), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm_terms(torch.from_numpy(x).cuda(), sa.pack_weights(s_d), e_d, t_d, q, N, K,
                              G, terms, 2, y)
    torch.cuda.synchronize()
    s, e, t = s_d.cpu().numpy(), e_d.cpu().numpy(), t_d.cpu().numpy()
    y_ref, a_ref = oracle.shiftadd_gemm_terms(x, s, e, t, G)
    assert (np.abs(y.cpu().numpy() - y_ref) / a_ref).max() <= 2e-3
    y_dense = x.astype(np.float64) @ bcq.reconstruct_terms(s, e, t, G).T
    assert np.abs(y_ref - y_dense).max() <= 1e-12 * a_ref.max()
    # the second term lowers the weight error
    s1, e1 = gpu_quantize(w, q, G, T)
    err1 = np.linalg.norm(bcq.reconstruct(s1, e1, G) - w)
    err2 = np.linalg.norm(bcq.reconstruct_terms(s, e, t, G) - w)
    assert err2 < err1
