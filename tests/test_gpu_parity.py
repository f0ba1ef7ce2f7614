"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars (fixed here, in the test):
* packing and unpacking: bit-exact;
* tables: |lut - lut_ref| <= 8 * 2^-24 * sum|x_chunk| (fp32 construction of a
  sum of 8 fp16 values), and entry 255-m == -entry m bitwise;
* the layer: max |y - y_ref| / sum|terms| <= 2e-3 per output (fp32
  accumulation of fp16 activations).  A second, stricter alarm at 1e-5 flags
  the error level fp32 tables should never reach.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads
from tests import _layout

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


def pack(signs_np):
    q, N, K = signs_np.shape
    s = dev(signs_np)
    p = sa.pack_weights(s)
    del s
    return p


def gemm(case, packed=None, exps=None, stream=None):
    q, N, K, G, B = case["q"], case["N"], case["K"], case["G"], case["B"]
    if packed is None:
        packed = pack(case["signs"])
    e = dev(case["exps"]) if exps is None else exps
    x = dev(case["x"])
    y = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm(x, packed, e, q, N, K, G, B, y, stream)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def check(y, y_ref, a_ref, what=""):
    y = y.astype(np.float64)
    assert np.isfinite(y).all(), what
    err = np.abs(y - y_ref)
    zero = a_ref == 0
    assert (err[zero] == 0).all(), what
    ratio = err[~zero] / a_ref[~zero] if (~zero).any() else np.zeros(1)
    worst = float(ratio.max()) if ratio.size else 0.0
    say(f"  {what}: max |y-y_ref|/sum|terms| = {worst:.3e}")
    assert worst <= TOL, what
    assert worst <= ALARM, f"{what}: error {worst:.3e} above the fp32-table alarm"
    return worst


# ----------------------------------------------------------------------------- packing

PACK_SHAPES = [(1, 1, 8), (3, 64, 128), (2, 65, 136), (3, 100, 256), (8, 130, 1040),
               (3, 768, 768), (2, 11008, 256), (3, 4096, 4096)]


@pytest.mark.parametrize("q,N,K", PACK_SHAPES)
def test_pack_bit_exact(q, N, K):
    say(f"pack q={q} N={N} K={K}")
    c = workloads.random_case(q, N, K, 8, 1, seed=q * 7 + N)
    p = pack(c["signs"])
    got = _layout.to_canonical(p.cpu().numpy(), q, N, K)
    assert np.array_equal(got, oracle.pack(c["signs"]))
    back = torch.empty((q, N, K), dtype=torch.int8, device="cuda")
    sa.sa_unpack_weights(p, q, N, K, back)
    torch.cuda.synchronize()
    assert np.array_equal(back.cpu().numpy(), c["signs"])


def test_pack_non_pm1_signs():
    say("pack non +-1 signs")
    rng = np.random.default_rng(3)
    s = rng.integers(-3, 4, (2, 70, 264)).astype(np.int8)
    p = pack(s)
    got = _layout.to_canonical(p.cpu().numpy(), 2, 70, 264)
    assert np.array_equal(got, oracle.pack(s))
    fixed = np.ones((1, 64, 128), np.int8)
    assert (pack(fixed).cpu().numpy() == 0xFF).all()
    assert (pack(-fixed).cpu().numpy() == 0x00).all()


# ----------------------------------------------------------------------------- tables

@pytest.mark.parametrize("K,B", [(8, 1), (64, 3), (768, 1), (4096, 2), (11008, 16), (256, 256)])
def test_build_lut(K, B):
    say(f"lut K={K} B={B}")
    c = workloads.random_case(1, 1, K, 8, B, seed=K + B, outlier_fraction=0.01)
    lut = torch.empty((B, K // 8, 256), dtype=torch.float32, device="cuda")
    sa.sa_build_lut(dev(c["x"]), K, B, lut)
    torch.cuda.synchronize()
    got = lut.cpu().numpy().astype(np.float64)
    ref = oracle.lut(c["x"])
    bound = 8 * 2.0 ** -24 * np.abs(c["x"].astype(np.float64)).reshape(B, K // 8, 8).sum(-1)
    assert (np.abs(got - ref) <= bound[..., None]).all()
    m = np.arange(256)
    g32 = lut.cpu().numpy()
    assert np.array_equal(g32[..., 255 - m], -g32[..., m])


def test_build_lut_hand_example():
    import json
    import os
    h = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))
    h = h["lut_chunk"]
    x = np.array([h["x"]], np.float16)
    lut = torch.empty((1, 1, 256), dtype=torch.float32, device="cuda")
    sa.sa_build_lut(dev(x), 8, 1, lut)
    torch.cuda.synchronize()
    t = lut.cpu().numpy()[0, 0]
    for key, val in h["entries"].items():
        assert t[int(key)] == val


# ----------------------------------------------------------------------------- the layer

SMALL = [
    # row kernel (group % 128 == 0, batch 1)
    (1, 1, 128, 128, 1), (3, 65, 256, 128, 1), (8, 64, 128, 128, 1), (3, 4097, 512, 128, 1),
    (2, 129, 9216, 384, 1), (3, 17, 4224, 128, 1),
    # row kernel, eight planes over a long input dimension (16 pieces)
    (8, 300, 65536, 128, 1),
    # row kernel, 16 waves taking two pieces at once (at most 256 workgroups,
    # several pieces): odd piece count with a one-block last piece, 256
    # workgroups, one group spanning both pieces
    (4, 1000, 8320, 128, 1), (3, 4096, 12288, 256, 1), (1, 16, 8192, 8192, 1),
    # ... with two row groups per workgroup (449..512 groups, several pieces)
    (3, 8000, 8320, 128, 1), (2, 8192, 8192, 256, 1),
    # row kernel, one piece and at most 256 row groups (one job per workgroup):
    # ragged last group, K below 4096 with idle blocks, groups of 256 to 1024
    (4, 4090, 3840, 256, 1), (1, 200, 1152, 384, 1), (2, 4096, 4096, 128, 1),
    (3, 31, 2048, 1024, 1),
    # decoder projections sharing an input run as one launch: q+k at q=2
    # (8192x4096), up+gate at q=3 (22016x4096)
    (2, 8192, 4096, 128, 1), (3, 22016, 4096, 128, 1),
    # batch kernel (group % 128 == 0, batch >= 2), 16- and 32-row workgroups
    (2, 300, 384, 128, 2), (3, 257, 1280, 256, 3), (4, 130, 768, 768, 5),
    (2, 1000, 4096, 128, 16), (3, 63, 2048, 128, 4), (2, 129, 1152, 384, 7),
    (3, 4100, 384, 384, 13), (8, 40, 384, 128, 6), (6, 300, 2176, 128, 9),
    # batch kernel, 64-row workgroups over three pieces
    (3, 4096, 2304, 128, 16),
    # batch kernel, 64-row workgroups (last piece and last tile ragged)
    (1, 28672, 1152, 128, 5), (2, 28000, 256, 256, 8),
    # batch kernel, 64-row workgroups, eight quads
    (1, 28600, 256, 128, 32),
    # batch kernel, every wave over 4, 8, 16 and 2 consecutive blocks
    (3, 1000, 4096, 128, 4), (2, 300, 8192, 128, 16), (4, 100, 16384, 128, 3),
    (1, 64, 2048, 128, 2),
    # generic kernel (any group % 8 == 0)
    (3, 100, 256, 8, 2), (1, 1, 8, 8, 1), (2, 257, 200, 40, 3), (3, 64, 1024, 64, 1),
    (4, 70, 96, 24, 1), (2, 33, 136, 136, 2),
]


@pytest.mark.parametrize("q,N,K,G,B", SMALL)
def test_gemm_small(q, N, K, G, B):
    say(f"gemm q={q} N={N} K={K} G={G} B={B} path={sa.sa_plan_gemm(q, N, K, G, B)['path']}")
    c = workloads.random_case(q, N, K, G, B, seed=1, exp_range=(-10, -2), outlier_fraction=0.01)
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], G)
    check(gemm(c), y_ref, a_ref, c["name"])


# whole-table K-slice layer: 1 to 8 slices; N from 5 rows (one partial 8-row
# job, waves without jobs) to 28672; ragged last job and last 64-row tile;
# groups of 128, 256 and 1024 columns; 1, 2, 3, 4 and 8 planes
KSLICE = [(3, 24576, 2048, 128), (1, 1000, 1024, 128), (4, 28672, 2048, 256),
          (2, 4100, 8192, 1024), (8, 300, 3072, 128), (3, 8, 1024, 128), (3, 5, 1024, 128)]


def gemm_kslice(case, packed=None, ws=None):
    q, N, K, G = case["q"], case["N"], case["K"], case["G"]
    if packed is None:
        packed = pack(case["signs"])
    if ws is None:
        ws = torch.full((sa.sa_kslice_workspace_bytes(N, K) // 4,), float("nan"),
                        dtype=torch.float32, device="cuda")
    y = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    sa.sa_shiftadd_gemm_kslice(dev(case["x"]), packed, dev(case["exps"]), q, N, K, G, y, ws)
    torch.cuda.synchronize()
    return y.cpu().numpy()[None, :]


@pytest.mark.parametrize("q,N,K,G", KSLICE)
def test_gemm_kslice(q, N, K, G):
    say(f"gemm kslice q={q} N={N} K={K} G={G}")
    c = workloads.random_case(q, N, K, G, 1, seed=3, exp_range=(-10, -2), outlier_fraction=0.01)
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], G)
    packed = pack(c["signs"])
    y = gemm_kslice(c, packed=packed)
    check(y, y_ref, a_ref, c["name"])
    # deterministic, and an exponent shift scales the output exactly
    assert np.array_equal(gemm_kslice(c, packed=packed), y)
    c2 = dict(c, exps=(c["exps"] + np.int8(3)).astype(np.int8))
    assert np.array_equal(gemm_kslice(c2, packed=packed), np.ldexp(y, 3).astype(np.float32))


def test_gemm_kslice_workspace_reuse():
    """One workspace for two layers in a row, the second smaller."""
    ws = torch.zeros(sa.sa_kslice_workspace_bytes(3000, 4096) // 4, dtype=torch.float32,
                     device="cuda")
    for q, N, K in ((3, 3000, 4096), (2, 777, 2048)):
        say(f"kslice workspace reuse q={q} N={N} K={K}")
        c = workloads.random_case(q, N, K, 128, 1, seed=4, exp_range=(-10, -2))
        y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128)
        check(gemm_kslice(c, ws=ws), y_ref, a_ref, c["name"])


@pytest.mark.parametrize("layer", [0, 1])
def test_gemm_kslice_70b_full_size(layer):
    """The two LLaMA-2-70B MLP shapes at full size, sampled rows (first and last
    64-row tiles and 512 seeded rows) against the oracle."""
    d = workloads.layer_inputs("llama2_70b_mlp", layer, 1)
    q, N, K, G = d["q"], d["N"], d["K"], d["G"]
    say(f"kslice full size {d['name']} q={q} N={N} K={K}")
    y = gemm_kslice(d)
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([np.arange(64), np.arange(N - 64, N),
                                     rng.choice(N, 512, replace=False)]))
    y_ref, a_ref = oracle.shiftadd_gemm(d["x"], d["signs"], d["exps"], G, rows=rows)
    check(y[:, rows], y_ref, a_ref, f"{d['name']} (sampled rows)")


# binary16 outputs: row kernel (one and several pieces), batch kernel, generic
# kernel; the last case's outputs exceed the binary16 range
F16_OUT = [(3, 4096, 4096, 128, 1, (-10, -2)), (3, 1000, 8320, 128, 1, (-10, -2)),
           (2, 300, 384, 128, 5, (-10, -2)), (4, 130, 768, 768, 16, (-10, -2)),
           (3, 100, 256, 8, 2, (-10, -2)), (3, 257, 1024, 128, 1, (10, 14))]


@pytest.mark.parametrize("q,N,K,G,B,er", F16_OUT)
def test_gemm_f16_output(q, N, K, G, B, er):
    say(f"gemm f16 output q={q} N={N} K={K} G={G} B={B} exps {er}")
    c = workloads.random_case(q, N, K, G, B, seed=6, exp_range=er, outlier_fraction=0.01)
    packed = pack(c["signs"])
    y32 = gemm(c, packed=packed)
    y16 = torch.full((B, N), float("nan"), dtype=torch.float16, device="cuda")
    sa.sa_shiftadd_gemm_f16(dev(c["x"]), packed, dev(c["exps"]), q, N, K, G, B, y16)
    torch.cuda.synchronize()
    y16 = y16.cpu().numpy()
    with np.errstate(over="ignore"):
        conv = y32.astype(np.float16)  # IEEE round to nearest even
    # the fp32 layer's result rounded to binary16, bit for bit
    assert np.array_equal(y16.view(np.uint16), conv.view(np.uint16))
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], G)
    if er[0] > 0:  # beyond the binary16 range: +-inf, within it: finite
        big, small = np.abs(y_ref) > 7e4, np.abs(y_ref) < 6e4
        assert big.any() and np.isinf(y16[big]).all() and np.isfinite(y16[small]).all()
        return
    err = np.abs(y16.astype(np.float64) - y_ref)
    assert (err <= TOL * a_ref + 2.0 ** -11 * np.abs(y_ref) + 2.0 ** -24).all(), c["name"]


@pytest.mark.parametrize("B", [2, 5, 8])
def test_batch_large_activations(B):
    """Activations near the top of the fp16 range in some blocks of some batch
    rows, next to fp16 subnormals and in a ragged last piece: table values reach
    about 2.4e5 and must stay exact to fp32 rounding."""
    say(f"batch large activations B={B}")
    c = workloads.random_case(3, 300, 2304, 128, B, seed=21)
    x = c["x"].astype(np.float32)
    x[0, 130:140] = 30000.0          # block 1, first batch row
    x[B - 1, 1000] = -60000.0        # block 7, last batch row
    x[B - 1, 1001:1004] = 3e-7       # fp16 subnormals next to it
    x[B // 2, 2200:2300] = 9000.0    # last (partial) piece, just above 8192
    c["x"] = x.astype(np.float16)
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128)
    check(gemm(c), y_ref, a_ref, "large activations")


@pytest.mark.parametrize("B", [1, 5])
def test_exps_at_odd_address(B):
    """Exponents may start at any byte address (the ABI asks no alignment)."""
    say(f"exps at odd address B={B}")
    c = workloads.random_case(3, 200, 1024, 128, B, seed=2, exp_range=(-10, -2))
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128)
    flat = c["exps"].reshape(-1)
    buf = torch.zeros(flat.size + 1, dtype=torch.int8, device="cuda")
    buf[1:] = dev(flat)
    e = buf[1:]
    assert e.data_ptr() % 2 == 1
    check(gemm(c, exps=e), y_ref, a_ref, "odd exps address")


def test_gemm_hand_example():
    import json
    import os
    h = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))
    h = h["layer"]
    c = dict(signs=np.array(h["signs"], np.int8), exps=np.array(h["exps"], np.int8),
             x=np.array(h["x"], np.float16), q=2, N=1, K=16, G=8, B=1)
    assert gemm(c).tolist() == h["y"]


def _layer_cases():
    return [pytest.param(key, li, id=f"{key}-{L.name}")
            for key, w in workloads.WORKLOADS.items() for li, L in enumerate(w.layers)]


@pytest.mark.parametrize("key,layer", _layer_cases())
def test_gemm_workload_full_size(key, layer):
    """Every named workload layer at its full size and every batch size it lists,
    in the launch configuration the benchmark times.  The oracle evaluates every
    output when that is cheap, else a seeded sample of rows that always includes
    the first and last 64-row tiles."""
    w = workloads.workload(key)
    d = workloads.layer_inputs_batches(key, layer, w.batches)
    q, N, K, G = d["q"], d["N"], d["K"], d["G"]
    packed = pack(d["signs"])
    e = dev(d["exps"])
    for B in w.batches:
        say(f"workload {d['name']} q={q} N={N} K={K} B={B} plan={sa.sa_plan_gemm(q, N, K, G, B)}")
        c = dict(d, x=d["x"][B], B=B)
        y = gemm(c, packed=packed, exps=e)
        if q * N * K * B <= 2e9:
            y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], G)
            check(y, y_ref, a_ref, f"{d['name']} B={B}")
        else:
            rng = np.random.default_rng(0)
            rows = np.unique(np.concatenate([np.arange(64), np.arange(N - 64, N),
                                             rng.choice(N, 512, replace=False)]))
            y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], G, rows=rows)
            check(y[:, rows], y_ref, a_ref, f"{d['name']} B={B} (sampled rows)")


@pytest.mark.parametrize("q,N,K,G,B", [(3, 500, 1024, 128, 1), (2, 257, 2048, 256, 4),
                                       (3, 100, 256, 8, 2), (2, 64, 768, 768, 2)])
@pytest.mark.parametrize("delta", [-5, 3])
def test_exact_shift_invariance_bitwise(q, N, K, G, B, delta):
    """Adding delta to every exponent scales y by exactly 2^delta."""
    say(f"shift q={q} N={N} K={K} G={G} B={B} delta={delta}")
    c = workloads.random_case(q, N, K, G, B, seed=5, exp_range=(-10, -2))
    packed = pack(c["signs"])
    y0 = gemm(c, packed=packed)
    c2 = dict(c, exps=(c["exps"] + np.int8(delta)).astype(np.int8))
    y1 = gemm(c2, packed=packed)
    assert np.array_equal(y1, np.ldexp(y0, delta).astype(np.float32))


def test_deterministic_and_back_to_back():
    say("determinism")
    c = workloads.random_case(3, 4096, 4096, 128, 1, seed=8, outlier_fraction=0.01)
    packed = pack(c["signs"])
    e = dev(c["exps"])
    x = dev(c["x"])
    ys = []
    for _ in range(5):
        y = torch.empty((1, 4096), dtype=torch.float32, device="cuda")
        sa.sa_shiftadd_gemm(x, packed, e, 3, 4096, 4096, 128, 1, y)
        ys.append(y)
    torch.cuda.synchronize()
    for y in ys[1:]:
        assert torch.equal(y, ys[0])


def test_non_default_stream():
    say("non-default stream")
    c = workloads.random_case(2, 700, 1536, 128, 3, seed=9)
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        packed = pack(c["signs"])
        y = gemm(c, packed=packed, stream=s)
    check(y, y_ref, a_ref, "side stream")


def test_alternating_shapes_on_one_stream():
    """Alternating shapes with different launch geometry (pieces, batch) on one
    stream: no call may depend on state left by another."""
    say("alternating shapes")
    cases = [workloads.random_case(3, 300, 4096, 128, 1, seed=10),
             workloads.random_case(2, 1000, 11008, 128, 2, seed=11),
             workloads.random_case(3, 300, 4096, 128, 5, seed=12)]
    refs = [oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128) for c in cases]
    for rep in range(2):
        for c, (y_ref, a_ref) in zip(cases, refs):
            check(gemm(c), y_ref, a_ref, f"rep {rep} {c['name']}")


@pytest.mark.parametrize("G", [128, 8])
def test_extreme_exponents(G):
    say(f"extreme exponents G={G}")
    c = workloads.random_case(3, 130, 512, G, 2, seed=13, exp_range=(-30, 30))
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], G)
    check(gemm(c), y_ref, a_ref, "exps in [-30, 30]")


def test_zero_activations_and_all_plus():
    say("zero x / all +1")
    c = workloads.random_case(3, 200, 1024, 128, 2, seed=14)
    z = dict(c, x=np.zeros_like(c["x"]))
    assert (gemm(z) == 0).all()
    p = dict(c, signs=np.ones_like(c["signs"]))
    y_ref, a_ref = oracle.shiftadd_gemm(p["x"], p["signs"], p["exps"], 128)
    check(gemm(p), y_ref, a_ref, "all +1")


def test_max_batch():
    say("batch 256")
    c = workloads.random_case(2, 70, 256, 128, 256, seed=15)
    y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128)
    check(gemm(c), y_ref, a_ref, "batch 256")


def test_binding_raises_on_bad_arguments():
    x = torch.zeros((1, 256), dtype=torch.float16, device="cuda")
    packed = torch.zeros(sa.sa_packed_bytes(3, 64, 256), dtype=torch.uint8, device="cuda")
    e = torch.zeros((3, 64, 2), dtype=torch.int8, device="cuda")
    ybig = torch.zeros(65, dtype=torch.float32, device="cuda")
    with pytest.raises(sa.SaError) as ei:
        sa.sa_shiftadd_gemm(x, packed, e, 3, 64, 256, 128, 1, ybig[1:])  # 4-byte offset
    assert ei.value.status == sa.SA_ERR_ALIGN
    with pytest.raises(ValueError):
        sa.sa_shiftadd_gemm(x, packed, e, 3, 64, 256, 128, 1, ybig)  # wrong numel
    with pytest.raises(sa.SaError):
        sa.sa_shiftadd_gemm(x, packed, e, 3, 64, 256, 96, 1, ybig[:64])


def test_small_then_large_row_counts():
    """Regression (an earlier design kept per-tile state between calls): a call
    with few rows and a large batch, then one with many rows, alternately."""
    say("small then large row counts")
    first = workloads.random_case(2, 1000, 4096, 128, 16, seed=16)
    second = workloads.random_case(3, 4097, 512, 128, 1, seed=17)
    for c in (first, second, first, second):
        y_ref, a_ref = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], 128)
        check(gemm(c), y_ref, a_ref, c["name"])
