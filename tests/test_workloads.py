"""The seeded generators: determinism, shapes, value sets and the stored goldens."""
import json
import os

import numpy as np
import pytest

import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_generator_determinism():
    a = workloads.random_case(3, 17, 256, 128, 2, seed=5)
    b = workloads.random_case(3, 17, 256, 128, 2, seed=5)
    c = workloads.random_case(3, 17, 256, 128, 2, seed=6)
    for k in ("signs", "exps", "x"):
        assert workloads.sha256(a[k]) == workloads.sha256(b[k])
        assert workloads.sha256(a[k]) != workloads.sha256(c[k])


def test_layer_inputs_properties():
    d = workloads.layer_inputs("opt125m_proj", 0, 1)
    assert d["signs"].shape == (3, 768, 768) and d["signs"].dtype == np.int8
    assert set(np.unique(d["signs"]).tolist()) == {-1, 1}
    assert d["exps"].shape == (3, 768, 6) and d["exps"].min() >= -8 and d["exps"].max() <= -2
    assert d["x"].shape == (1, 768) and d["x"].dtype == np.float16
    # fair coins: the +1 fraction is close to 1/2
    assert abs((d["signs"] > 0).mean() - 0.5) < 0.01


def test_weights_do_not_depend_on_batch():
    a = workloads.layer_inputs("llama2_7b_mlp_q2", 1, 1)
    b = workloads.layer_inputs("llama2_7b_mlp_q2", 1, 4)
    assert np.array_equal(a["exps"], b["exps"])
    assert workloads.sha256(a["signs"]) == workloads.sha256(b["signs"])
    assert b["x"].shape == (4, 11008)


def test_outlier_channels():
    d = workloads.layer_inputs("llama2_7b_attn", 0, 1)
    idx = d["outlier_channels"]
    assert idx.size == 41 and np.unique(idx).size == 41  # round(0.01 * 4096), no repeats
    x = np.abs(d["x"].astype(np.float64))[0]
    rest = np.setdiff1d(np.arange(4096), idx)
    assert x[rest].max() < 6.0  # N(0,1) elsewhere
    assert np.median(x[idx]) > 5.0  # 20 * |N(0,1)| has median ~13.5
    assert d["exps"].min() >= -10 and d["exps"].max() <= -3


def test_copies_are_distinct():
    a = workloads.layer_inputs("opt125m_proj", 0, 1, copy=0)
    b = workloads.layer_inputs("opt125m_proj", 0, 1, copy=1)
    assert workloads.sha256(a["signs"]) != workloads.sha256(b["signs"])


def test_mixed_bits():
    qs = workloads.mixed_bits(0)
    assert len(qs) == 7 and sum(qs) == 21 and set(qs) <= {2, 3, 4}
    w = workloads.workload("llama2_7b_layer_set")
    assert [L.q for L in w.layers] == qs and w.depth == 32


def test_golden_small_cases(oracle_mod):
    with open(os.path.join(GOLDEN, "oracle_small_cases.json")) as f:
        g = json.load(f)
    assert g["mixed_bits_7b_layer_set"] == workloads.mixed_bits(0)
    for case in g["cases"]:
        s = case["spec"]
        c = workloads.random_case(s["q"], s["N"], s["K"], s["G"], s["B"], seed=s["seed"],
                                  exp_range=tuple(s["exp_range"]),
                                  outlier_fraction=s["outlier_fraction"])
        for k in ("signs", "exps", "x"):
            assert workloads.sha256(c[k]) == case["sha256"][k], k
        y, a = oracle_mod.shiftadd_gemm(c["x"], c["signs"], c["exps"], s["G"])
        assert [[v.hex() for v in row] for row in y] == case["y"]
        assert [[v.hex() for v in row] for row in a] == case["absterm"]


def test_layer_inputs_batches_matches_single_draws():
    d = workloads.layer_inputs_batches("llama2_7b_attn", 0, (1, 3))
    for B in (1, 3):
        e = workloads.layer_inputs("llama2_7b_attn", 0, B)
        assert np.array_equal(d["x"][B], e["x"])
        assert np.array_equal(d["exps"], e["exps"])
    assert workloads.sha256(d["signs"]) == workloads.sha256(e["signs"])
