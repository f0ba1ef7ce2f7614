"""Seeded synthetic inputs for the shift-add linear layer.

This module is shared by the CPU oracle (tests, cpu baseline) and the GPU path
(tests, bench).  It only draws random numbers: it holds none of the method's
arithmetic (no bit packing, no table construction, no scaling).

What is drawn, per layer of shape N x K with q binary planes and group size G
(ShiftAddLLM, Sec. 3 "Binary-coding Quantization" and Sec. 4.1):

* ``signs``  int8 ``[q][N][K]`` in {-1, +1}: the binary matrices b_i, each entry
  an independent fair coin (the Bernoulli(0.5) planes of the synthetic layers),
  taken from the bits of uniformly random bytes.
* ``exps``   int8 ``[q][N][K/G]``: the power-of-two exponents P of the scaling
  factors 2^P (Eq. 2), uniform over an inclusive integer range.  The sign of a
  scaling factor is assumed folded into the plane, so only magnitudes remain.
* ``x``      fp16 ``[B][K]``: activations N(0, 1); for the workloads with
  outliers, round(0.01 K) channels (the same for every batch row, drawn without
  replacement) are multiplied by 20 before the cast to fp16.

For the offline reparameterization (full-precision weights -> planes and
exponents), ``fp_weights`` draws fp32 ``[N][K]`` stand-ins for pretrained
projection weights: N(0, scale^2) scaled per row by a log-normal factor
(exp(N(0, 0.25^2))), with a fraction of entries multiplied by
``outlier_scale`` (the heavy tail of LLM weights).

Draw order per layer is fixed: signs, exps, x, outlier channels, from
``numpy.random.default_rng(SeedSequence([seed, config_id, layer_id]))``.

The paper's own evaluation data (WikiText-2, zero-shot suites, pretrained
OPT/LLaMA weights) is not available; these layers reproduce only the shapes,
bit widths and group sizes of the paper's OPT/LLaMA projections.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "Layer",
    "Workload",
    "WORKLOADS",
    "workload",
    "layer_inputs",
    "layer_inputs_batches",
    "random_case",
    "mixed_bits",
    "sha256",
    "fp_weights",
    "colwise_case",
    "blockwise_case",
    "terms_case",
    "layer_coins_batches",
]


@dataclasses.dataclass(frozen=True)
class Layer:
    name: str
    N: int  # output rows
    K: int  # input columns (reduction dimension)
    q: int  # binary planes


@dataclasses.dataclass(frozen=True)
class Workload:
    key: str
    config_id: int
    description: str
    layers: Tuple[Layer, ...]
    group: int
    exp_range: Tuple[int, int]  # inclusive
    outlier_fraction: float  # fraction of channels scaled by outlier_scale
    outlier_scale: float
    batches: Tuple[int, ...]
    depth: int = 1  # decoder depth the layer set is replicated over


def mixed_bits(seed: int = 0, n_layers: int = 7, choices=(2, 3, 4), mean: int = 3) -> List[int]:
    """Per-layer bit widths for the mixed-precision 7B layer set.

    Draw n_layers values uniformly from ``choices`` and redraw until their mean
    over layers equals ``mean`` (the budget of Eq. 4 counts layers, not
    parameters).
    """
    rng = np.random.default_rng(np.random.SeedSequence([seed, 4, 999]))
    target = mean * n_layers
    while True:
        qs = [int(v) for v in rng.choice(np.asarray(choices), size=n_layers)]
        if sum(qs) == target:
            return qs


def _layer_set(seed: int = 0) -> Tuple[Layer, ...]:
    names = ["q_proj", "k_proj", "v_proj", "o_proj", "up_proj", "gate_proj", "down_proj"]
    shapes = [(4096, 4096)] * 4 + [(11008, 4096)] * 2 + [(4096, 11008)]
    qs = mixed_bits(seed)
    return tuple(Layer(n, N, K, q) for n, (N, K), q in zip(names, shapes, qs))


WORKLOADS: Dict[str, Workload] = {
    w.key: w
    for w in (
        Workload(
            "opt125m_proj", 0,
            "OPT-125M-shaped projection 768x768, q=3, G=128, exps in [-8,-2], x ~ N(0,1)",
            (Layer("proj", 768, 768, 3),), 128, (-8, -2), 0.0, 1.0, (1,)),
        Workload(
            "llama2_7b_attn", 1,
            "LLaMA-2-7B attention projection 4096x4096, q=3, G=128, exps in [-10,-3], "
            "x ~ N(0,1) with 1% of channels x20",
            (Layer("attn_proj", 4096, 4096, 3),), 128, (-10, -3), 0.01, 20.0, (1,)),
        Workload(
            "llama2_7b_mlp_q2", 2,
            "LLaMA-2-7B MLP pair at q=2: up/gate 11008x4096 and down 4096x11008, G=128, "
            "exps in [-10,-3], x ~ N(0,1)",
            (Layer("up_gate", 11008, 4096, 2), Layer("down", 4096, 11008, 2)),
            128, (-10, -3), 0.0, 1.0, (1, 4, 16)),
        Workload(
            "llama2_70b_mlp", 3,
            "LLaMA-2-70B-shaped MLP: 28672x8192 and 8192x28672, q=3, G=128, exps in [-12,-3], "
            "x ~ N(0,1)",
            (Layer("up", 28672, 8192, 3), Layer("down", 8192, 28672, 3)),
            128, (-12, -3), 0.0, 1.0, (1, 8)),
        Workload(
            "llama2_7b_layer_set", 4,
            "LLaMA-2-7B decoder linear layers (q,k,v,o 4096x4096; up, gate 11008x4096; "
            "down 4096x11008) with per-layer q in {2,3,4}, mean 3 over layers, G=128, "
            "exps in [-10,-3], x ~ N(0,1) with 1% of channels x20, replicated over 32 layers",
            _layer_set(0), 128, (-10, -3), 0.01, 20.0, (1, 4, 8, 16), depth=32),
        Workload(
            "llama2_70b_mlp_shard8", 5,
            "One GPU's shard of the LLaMA-2-70B-shaped MLP split 8 ways: up 3584x8192 "
            "(rows split) and down 8192x3584 (columns split), q=3, G=128, exps in [-12,-3], "
            "x ~ N(0,1)",
            (Layer("up_shard", 3584, 8192, 3), Layer("down_shard", 8192, 3584, 3)),
            128, (-12, -3), 0.0, 1.0, (1, 8)),
    )
}


def workload(key: str) -> Workload:
    return WORKLOADS[key]


def sha256(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def _draw_weights(rng: np.random.Generator, q: int, N: int, K: int, G: int,
                  exp_range: Tuple[int, int]):
    # signs: fair coins mapped to {-1, +1}; the coins are the bits of uniformly
    # random bytes (8 coins per byte drawn)
    coins = np.unpackbits(rng.integers(0, 256, size=(q, N, K // 8), dtype=np.uint8),
                          axis=-1, bitorder="little")
    signs = coins.view(np.int8)
    signs *= 2
    signs -= 1
    exps = rng.integers(exp_range[0], exp_range[1] + 1, size=(q, N, K // G), dtype=np.int8)
    return signs, exps


def _draw_x(rng: np.random.Generator, K: int, B: int, outlier_fraction: float,
            outlier_scale: float):
    x = rng.standard_normal((B, K))
    n_out = int(round(outlier_fraction * K))
    idx = np.zeros(0, dtype=np.int64)
    if n_out > 0:
        idx = rng.choice(K, size=n_out, replace=False)
        x[:, idx] *= outlier_scale
    return x.astype(np.float16), np.sort(idx)


def _draw(rng, q, N, K, G, B, exp_range, outlier_fraction, outlier_scale):
    signs, exps = _draw_weights(rng, q, N, K, G, exp_range)
    x16, idx = _draw_x(rng, K, B, outlier_fraction, outlier_scale)
    return signs, exps, x16, idx


def layer_inputs(key: str, layer: int, batch: int, seed: int = 0, copy: int = 0) -> dict:
    """Inputs of one layer of a named workload.

    ``copy`` selects a distinct replica of the layer (another decoder depth in the
    layer set, or another weight copy that benchmarks rotate through so that the
    last-level cache cannot serve the weights).  Weights do not depend on
    ``batch``: the same seed gives the same planes and exponents at every batch.
    """
    w = WORKLOADS[key]
    L = w.layers[layer]
    layer_id = layer + 1000 * copy
    rng = np.random.default_rng(np.random.SeedSequence([seed, w.config_id, layer_id]))
    signs, exps, x16, idx = _draw(rng, L.q, L.N, L.K, w.group, batch, w.exp_range,
                                  w.outlier_fraction, w.outlier_scale)
    return dict(signs=signs, exps=exps, x=x16, outlier_channels=idx,
                q=L.q, N=L.N, K=L.K, G=w.group, B=batch,
                name=f"{key}/{L.name}", seed=seed, copy=copy)


def layer_inputs_batches(key: str, layer: int, batches: Sequence[int], seed: int = 0,
                         copy: int = 0) -> dict:
    """One draw of a layer's weights with the activations of several batch sizes.

    ``x[B]`` equals ``layer_inputs(key, layer, B, seed, copy)["x"]``: the
    activations are drawn from the generator state right after the weights.
    """
    w = WORKLOADS[key]
    L = w.layers[layer]
    rng = np.random.default_rng(np.random.SeedSequence([seed, w.config_id, layer + 1000 * copy]))
    signs, exps = _draw_weights(rng, L.q, L.N, L.K, w.group, w.exp_range)
    state = rng.bit_generator.state
    xs = {}
    for B in batches:
        rng.bit_generator.state = state
        xs[B] = _draw_x(rng, L.K, B, w.outlier_fraction, w.outlier_scale)[0]
    return dict(signs=signs, exps=exps, x=xs, q=L.q, N=L.N, K=L.K, G=w.group,
                name=f"{key}/{L.name}", seed=seed, copy=copy)


def random_case(q: int, N: int, K: int, G: int, B: int, seed: int = 0,
                exp_range: Tuple[int, int] = (-8, -2), outlier_fraction: float = 0.0,
                outlier_scale: float = 20.0, x_scale: float = 1.0) -> dict:
    """A seeded layer of arbitrary shape (parity and edge cases)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 100, q, N, K, G, B]))
    signs, exps, x16, idx = _draw(rng, q, N, K, G, B, exp_range, outlier_fraction,
                                  outlier_scale)
    if x_scale != 1.0:
        x16 = (x16.astype(np.float64) * x_scale).astype(np.float16)
    return dict(signs=signs, exps=exps, x=x16, outlier_channels=idx, q=q, N=N, K=K, G=G, B=B,
                name=f"case(q={q},N={N},K={K},G={G},B={B},seed={seed})", seed=seed, copy=0)



def fp_weights(N: int, K: int, seed: int = 0, scale: float = 0.02,
               outlier_fraction: float = 1e-3, outlier_scale: float = 10.0) -> np.ndarray:
    """Seeded fp32 weights [N][K] for the offline reparameterization.

    Draw order: per-row factors, the Gaussian body, then the outlier positions
    (uniform over the N*K entries, with replacement; a repeated position is
    scaled once)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 200, N, K]))
    rows = np.exp(0.25 * rng.standard_normal((N, 1)))
    w = rng.standard_normal((N, K)) * (scale * rows)
    n_out = int(round(outlier_fraction * N * K))
    if n_out > 0:
        idx = np.unique(rng.integers(0, N * K, size=n_out))
        w.reshape(-1)[idx] *= outlier_scale
    return w.astype(np.float32)


def colwise_case(q: int, N: int, K: int, B: int, seed: int = 0,
                 exp_range: Tuple[int, int] = (-10, -3), outlier_fraction: float = 0.01,
                 outlier_scale: float = 20.0, copy: int = 0) -> dict:
    """A seeded layer with column-wise factors ("Acc."): signs [q][N][K] as for
    the row-wise layers, exponents int8 [q][K] (one per plane and column,
    uniform over the inclusive range), fp16 activations [B][K] with outlier
    channels.  Draw order: signs, column exponents, x, outlier channels."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 300, q, N, K, B, copy]))
    coins = np.unpackbits(rng.integers(0, 256, size=(q, N, K // 8), dtype=np.uint8),
                          axis=-1, bitorder="little")
    signs = coins.view(np.int8)
    signs *= 2
    signs -= 1
    col_exps = rng.integers(exp_range[0], exp_range[1] + 1, size=(q, K), dtype=np.int8)
    x16, idx = _draw_x(rng, K, B, outlier_fraction, outlier_scale)
    return dict(signs=signs, col_exps=col_exps, x=x16, outlier_channels=idx, q=q, N=N, K=K,
                B=B, name=f"colwise(q={q},N={N},K={K},B={B},seed={seed})", seed=seed, copy=copy)


def blockwise_case(q: int, N: int, K: int, B: int, row_block: int, seed: int = 0,
                   exp_range: Tuple[int, int] = (-10, -3), outlier_fraction: float = 0.01,
                   outlier_scale: float = 20.0, copy: int = 0) -> dict:
    """A seeded layer with block-wise factors ("Lat."): signs [q][N][K], one
    int8 exponent per plane, block of ``row_block`` rows and 8 columns
    ([q][ceil(N / row_block)][K / 8], uniform over the inclusive range), fp16
    activations [B][K] with outlier channels.  Draw order: signs, exponents,
    x, outlier channels."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 400, q, N, K, B, row_block, copy]))
    coins = np.unpackbits(rng.integers(0, 256, size=(q, N, K // 8), dtype=np.uint8),
                          axis=-1, bitorder="little")
    signs = coins.view(np.int8)
    signs *= 2
    signs -= 1
    NB = -(-N // row_block)
    blk_exps = rng.integers(exp_range[0], exp_range[1] + 1, size=(q, NB, K // 8), dtype=np.int8)
    x16, idx = _draw_x(rng, K, B, outlier_fraction, outlier_scale)
    return dict(signs=signs, blk_exps=blk_exps, row_block=row_block, x=x16,
                outlier_channels=idx, q=q, N=N, K=K, B=B,
                name=f"blockwise(q={q},N={N},K={K},B={B},rb={row_block},seed={seed})",
                seed=seed, copy=copy)


def terms_case(q: int, N: int, K: int, G: int, B: int, T: int, seed: int = 0,
               exp_range: Tuple[int, int] = (-10, -3), outlier_fraction: float = 0.01,
               outlier_scale: float = 20.0, copy: int = 0) -> dict:
    """A seeded layer with additive power-of-two factors (Eq. 2, T terms):
    signs [q][N][K]; exps int8 [q][N][K/G][T] where term t is drawn below the
    previous one (term 0 uniform over the range, term t = term t-1 minus 1..3,
    as a greedy residual expansion would give); term signs int8 [q][N][K/G][T]:
    term 0 is +1 (its sign is folded into the plane), later terms are +-1 or, one
    time in eight, 0 (no term).  Draw order: signs, exps, term signs, x,
    outlier channels."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 500, q, N, K, G, B, T, copy]))
    coins = np.unpackbits(rng.integers(0, 256, size=(q, N, K // 8), dtype=np.uint8),
                          axis=-1, bitorder="little")
    signs = coins.view(np.int8)
    signs *= 2
    signs -= 1
    NG = K // G
    e0 = rng.integers(exp_range[0], exp_range[1] + 1, size=(q, N, NG))
    exps = np.empty((T, q, N, NG), dtype=np.int8)
    exps[0] = e0
    for t in range(1, T):
        e0 = e0 - rng.integers(1, 4, size=(q, N, NG))
        exps[t] = e0
    tsg = rng.choice(np.array([-1, 1, 1, 1, -1, 1, -1, 0], dtype=np.int8), size=(T, q, N, NG))
    tsg[0] = 1
    exps = np.ascontiguousarray(exps.transpose(1, 2, 3, 0))   # term index last
    tsg = np.ascontiguousarray(tsg.transpose(1, 2, 3, 0))
    x16, idx = _draw_x(rng, K, B, outlier_fraction, outlier_scale)
    return dict(signs=signs, exps=exps, term_signs=tsg, x=x16, outlier_channels=idx, q=q, N=N,
                K=K, G=G, B=B, T=T, name=f"terms(q={q},N={N},K={K},G={G},B={B},T={T})",
                seed=seed, copy=copy)


def layer_coins_batches(key: str, layer: int, batches: Sequence[int], seed: int = 0,
                        copy: int = 0) -> dict:
    """``layer_inputs_batches`` without the unpacking of the sign bits: the same
    draws, with the planes as the drawn bytes (``coins`` uint8 [q][N][K/8]; bit
    j of byte c, little-endian, is the coin of column 8c+j, 1 -> +1).  For
    benchmarks that unpack on the device."""
    w = WORKLOADS[key]
    L = w.layers[layer]
    rng = np.random.default_rng(np.random.SeedSequence([seed, w.config_id, layer + 1000 * copy]))
    coins = rng.integers(0, 256, size=(L.q, L.N, L.K // 8), dtype=np.uint8)
    exps = rng.integers(w.exp_range[0], w.exp_range[1] + 1, size=(L.q, L.N, L.K // w.group),
                        dtype=np.int8)
    state = rng.bit_generator.state
    xs = {}
    for B in batches:
        rng.bit_generator.state = state
        xs[B] = _draw_x(rng, L.K, B, w.outlier_fraction, w.outlier_scale)[0]
    return dict(coins=coins, exps=exps, x=xs, q=L.q, N=L.N, K=L.K, G=w.group,
                name=f"{key}/{L.name}", seed=seed, copy=copy)
