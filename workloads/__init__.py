"""Seeded synthetic inputs for the NVFP4 linear-layer workloads.

This module only draws random numbers and rounds them to BF16; it holds none
of the method's arithmetic, and both the GPU library's tests/benchmark and the
CPU oracle take their inputs from here.

Shapes follow the denoisers the paper trains (Sec. 4.1 and the hyper-parameter
table of the appendix: SANA at 1024^2, FLUX.1 and SD3.5-Large; rollouts per
GPU from the Best-of-N setting).  The paper's prompts, weights and reward
models are not used: activations and weights are random with the value
distributions listed in ``WORKLOADS``.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Layer:
    name: str
    N: int          # output features
    K: int          # input features (multiple of 16)
    x_dist: str     # activation distribution, see draw_activations
    index: int      # layer index used in the seed


@dataclass(frozen=True)
class Workload:
    name: str
    config_id: int
    M: int                       # tokens (rollouts x tokens per rollout)
    layers: tuple
    w_sigma: float
    description: str = ""
    extra: dict = field(default_factory=dict)


WORKLOADS = {
    "single-1152": Workload(
        "single-1152", 0, 128,
        (Layer("linear", 1152, 1152, "outlier4x20", 0),), 0.02,
        "one linear, M=128, K=N=1152; X ~ N(0,1) with 4 outlier channels x20"),
    "sana-1.6b": Workload(
        "sana-1.6b", 1, 8 * 1024,
        (Layer("qkv", 6720, 2240, "t3_1pct", 0), Layer("out", 2240, 2240, "t3_1pct", 1),
         Layer("up", 5600, 2240, "t3_1pct", 2), Layer("down", 2240, 5600, "t3_1pct", 3)),
        0.02, "8 rollouts x 1024 image tokens, hidden 2240, MLP 5600; "
              "X ~ N(0,1) with 1% of elements Student-t(3)"),
    "flux-12b": Workload(
        "flux-12b", 2, 4 * (4096 + 512),
        (Layer("qkv", 9216, 3072, "normal", 0), Layer("out", 3072, 3072, "normal", 1),
         Layer("up", 12288, 3072, "normal", 2), Layer("down", 3072, 12288, "gelu", 3)),
        0.015, "4 rollouts x (4096 image + 512 text) tokens, hidden 3072, MLP 12288; "
               "X ~ N(0,1), MLP-down input GELU(N(0,1))"),
    "sd35-large": Workload(
        "sd35-large", 3, 6 * (4096 + 333),
        (Layer("qkv", 7296, 2432, "rowscale", 0), Layer("up", 9728, 2432, "rowscale", 1),
         Layer("down", 2432, 9728, "rowscale", 2)),
        0.02, "6 rollouts x (4096 image + 333 text) tokens, hidden 2432, MLP 9728; "
              "X ~ N(0,1) x per-token 10^U(-1,1)"),
}

ROLE_X, ROLE_W, ROLE_BIAS = 1, 2, 3

#: Rows per independently seeded chunk: chunk c of a tensor with seed s draws
#: from PCG64(SeedSequence(s).spawn(n_chunks)[c]), so tensors are generated in
#: parallel and any row range can be regenerated on its own.
CHUNK_ROWS = 256
_THREADS = max(1, min(16, os.cpu_count() or 1))


def seed_for(config_id: int, layer_index: int, role: int) -> int:
    return 1000 * config_id + 10 * layer_index + role


def rng(seed) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def f32_to_bf16_bits(a) -> np.ndarray:
    """Round float32 to BF16 bit patterns (nearest, ties to even); finite only."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    t = u >> np.uint32(16)
    t &= np.uint32(1)
    t += np.uint32(0x7FFF)
    t += u
    t >>= np.uint32(16)
    return t.astype(np.uint16)


def _gelu_erf(z: np.ndarray) -> np.ndarray:
    from scipy.special import erf
    return (np.float32(0.5) * z * (np.float32(1.0) + erf(z * np.float32(0.70710677)))).astype(np.float32)


def _draw_chunk(dist: str, g: np.random.Generator, rows: int, K: int, cols) -> np.ndarray:
    if dist == "normal":
        x = g.standard_normal((rows, K), dtype=np.float32)
    elif dist == "outlier4x20":
        x = g.standard_normal((rows, K), dtype=np.float32)
        x[:, cols] *= np.float32(20.0)
    elif dist == "t3_1pct":
        x = g.standard_normal((rows, K), dtype=np.float32)
        mask = g.random((rows, K), dtype=np.float32) < np.float32(0.01)
        x[mask] = g.standard_t(3, size=int(mask.sum())).astype(np.float32)
    elif dist == "gelu":
        x = _gelu_erf(g.standard_normal((rows, K), dtype=np.float32))
    elif dist == "rowscale":
        x = g.standard_normal((rows, K), dtype=np.float32)
        x *= np.power(np.float32(10.0), g.uniform(-1.0, 1.0, size=(rows, 1))).astype(np.float32)
    elif dist == "uniform":
        x = g.uniform(-1.0, 1.0, size=(rows, K)).astype(np.float32)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return f32_to_bf16_bits(x)


def draw_activations(dist: str, rows: int, K: int, seed: int, row_range=None) -> np.ndarray:
    """BF16 bit patterns [rows, K] of the named activation distribution; with
    ``row_range=(r0, r1)`` only those rows of the same tensor."""
    r0, r1 = (0, rows) if row_range is None else row_range
    if not 0 <= r0 <= r1 <= rows:
        raise ValueError(f"row_range {(r0, r1)} outside [0, {rows}]")
    n_chunks = max(1, -(-rows // CHUNK_ROWS))
    seeds = np.random.SeedSequence(seed).spawn(n_chunks)
    cols = rng(seed).choice(K, size=min(4, K), replace=False) if dist == "outlier4x20" else None
    out = np.empty((r1 - r0, K), dtype=np.uint16)
    c0, c1 = r0 // CHUNK_ROWS, -(-r1 // CHUNK_ROWS)

    def work(c):
        lo, hi = c * CHUNK_ROWS, min(rows, (c + 1) * CHUNK_ROWS)
        blk = _draw_chunk(dist, rng(seeds[c]), hi - lo, K, cols)
        a, b = max(lo, r0), min(hi, r1)
        out[a - r0:b - r0] = blk[a - lo:b - lo]

    if c1 - c0 > 1:
        with ThreadPoolExecutor(_THREADS) as ex:
            list(ex.map(work, range(c0, c1)))
    elif c1 > c0:
        work(c0)
    return out


def draw_weights(N: int, K: int, sigma: float, seed: int, row_range=None) -> np.ndarray:
    """BF16 bit patterns of an [N, K] weight ~ N(0, sigma^2)."""
    r0, r1 = (0, N) if row_range is None else row_range
    if not 0 <= r0 <= r1 <= N:
        raise ValueError(f"row_range {(r0, r1)} outside [0, {N}]")
    n_chunks = max(1, -(-N // CHUNK_ROWS))
    seeds = np.random.SeedSequence(seed).spawn(n_chunks)
    out = np.empty((r1 - r0, K), dtype=np.uint16)
    c0, c1 = r0 // CHUNK_ROWS, -(-r1 // CHUNK_ROWS)

    def work(c):
        lo, hi = c * CHUNK_ROWS, min(N, (c + 1) * CHUNK_ROWS)
        w = rng(seeds[c]).standard_normal((hi - lo, K), dtype=np.float32)
        w *= np.float32(sigma)
        blk = f32_to_bf16_bits(w)
        a, b = max(lo, r0), min(hi, r1)
        out[a - r0:b - r0] = blk[a - lo:b - lo]

    if c1 - c0 > 1:
        with ThreadPoolExecutor(_THREADS) as ex:
            list(ex.map(work, range(c0, c1)))
    elif c1 > c0:
        work(c0)
    return out


def draw_bias(N: int, sigma: float, seed: int) -> np.ndarray:
    g = rng(seed)
    return f32_to_bf16_bits(g.standard_normal(N, dtype=np.float32) * np.float32(sigma))


def layer_inputs(workload: Workload, layer: Layer, rows: int | None = None, bias: bool = True):
    """(x_bits [rows, K], w_bits [N, K], bias_bits [N] or None) for one layer;
    ``rows`` defaults to the workload's M."""
    rows = workload.M if rows is None else rows
    x = draw_activations(layer.x_dist, rows, layer.K,
                         seed_for(workload.config_id, layer.index, ROLE_X))
    w = draw_weights(layer.N, layer.K, workload.w_sigma,
                     seed_for(workload.config_id, layer.index, ROLE_W))
    b = (draw_bias(layer.N, workload.w_sigma, seed_for(workload.config_id, layer.index, ROLE_BIAS))
         if bias else None)
    return x, w, b
