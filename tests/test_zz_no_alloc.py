"""sa_importance_criterion_noalloc (the criterion of Eq. 3 with its partial sums
in the library's fixed device array instead of a caller workspace) against
sa_importance_criterion, through the C ABI.

Bar (fixed here): the same kernels on the same inputs, so the three fp64
results are bit-identical to the workspace entry point's; and, as for that
entry point, relative 1e-12 against a numpy fp64 evaluation of C = ||IS||_F
STD(IS)^2.  Two calls in a row, the second on a smaller input, check that the
array's contents from one call do not leak into the next.
"""
import ctypes
import sys

import numpy as np
import pytest

import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - CPU-only environment
    pytest.skip("no GPU", allow_module_level=True)
sa = pytest.importorskip("paper_2406_05981_amd.shiftadd")


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def with_workspace(w, d, N, K):
    out = torch.full((3,), float("nan"), dtype=torch.float64, device="cuda")
    ws = torch.empty(sa.lib.sa_importance_workspace(), dtype=torch.uint8, device="cuda")
    sa.sa_importance_criterion(w, N, K, d, out, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def without_workspace(w, d, N, K):
    out = torch.full((3,), float("nan"), dtype=torch.float64, device="cuda")
    st = sa.lib.sa_importance_criterion_noalloc(
        ctypes.c_void_p(w.data_ptr()), N, K, ctypes.c_void_p(d.data_ptr()),
        ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, sa.sa_status_string(st)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def case(N, K, seed):
    w = workloads.fp_weights(N, K, seed=seed)
    d = np.random.default_rng(seed + 1).uniform(0.01, 1.0, K)
    return w, d


def reference(w, d):
    IS = w.astype(np.float64) / d[None, :]
    return np.array([np.linalg.norm(IS) * IS.std() ** 2, np.linalg.norm(IS), IS.std()])


def test_noalloc_matches_workspace_entry_point_twice():
    for (N, K, seed) in [(1500, 2048, 7), (37, 300, 8)]:   # the second call is smaller
        say(f"criterion without workspace N={N} K={K}")
        w, d = case(N, K, seed)
        wt, dt = torch.from_numpy(w).cuda(), torch.from_numpy(d).cuda()
        got = without_workspace(wt, dt, N, K)
        ref = with_workspace(wt, dt, N, K)
        assert np.isfinite(got).all()
        assert np.array_equal(got, ref)
        assert np.allclose(got, reference(w, d), rtol=1e-12, atol=0)


def test_noalloc_rejects_bad_arguments():
    w = torch.zeros(4, dtype=torch.float32, device="cuda")
    d = torch.ones(2, dtype=torch.float64, device="cuda")
    out = torch.zeros(4, dtype=torch.float64, device="cuda")
    f = sa.lib.sa_importance_criterion_noalloc
    P = ctypes.c_void_p
    assert f(None, 2, 2, P(d.data_ptr()), P(out.data_ptr()), None) == -1       # SA_ERR_NULL
    assert f(P(w.data_ptr()), 0, 2, P(d.data_ptr()), P(out.data_ptr()), None) == -2  # SA_ERR_SHAPE
    assert f(P(w.data_ptr()), 1 << 21, 1 << 20, P(d.data_ptr()), P(out.data_ptr()), None) == -2
    assert f(P(w.data_ptr()), 2, 2, P(d.data_ptr()), P(out.data_ptr() + 4), None) == -5  # SA_ERR_ALIGN
