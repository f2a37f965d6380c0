"""CPU oracle of the synthetic Stage-1 rollout loop (test infrastructure:
only tests/ and bench.py's cpu_baseline leg may import it).

Stage 1 of the paper's two-stage framework (Sec. 3.4): roll out with the
quantized exploration model, score every rollout, keep the highest- and
lowest-rewarded ones.  This is the same loop as the GPU harness, written
plainly in float64 numpy with a BF16 rounding wherever the GPU stores a BF16
tensor:

    h = bf16(rmsnorm(x))                 x * (mean(x^2) + 1e-6)^-1/2
    qkv = linear(h)                      NVFP4 / MXFP4 oracle, or exact BF16 product
    a = bf16(softmax(q k^T / sqrt(d)) v) per rollout and head
    x = bf16(x + linear(a))
    h = bf16(rmsnorm(x)); u = bf16(gelu_tanh(linear(h))); x = bf16(x + linear(u))
    Euler: x = bf16(x + (1/T)(blocks(x) - x))
    reward_i = mean over the rollout's tokens of <x, u_dir>

linear(x) = bf16(x W^T + bias) with the format's quantization of x (and W,
quantized once by the same oracle).  The elementwise ops and the attention
are ordinary float64; only the linears carry the method's arithmetic.
"""
from __future__ import annotations

import numpy as np

from . import nvfp4 as O

EPS = 1e-6


def bf16_round(v):
    return O.bf16_bits_to_f32(O.f64_to_bf16_bits_rne(np.asarray(v, dtype=np.float64))).astype(np.float64)


def bits(v):
    return O.f64_to_bf16_bits_rne(np.asarray(v, dtype=np.float64))


def prepare(backend, w_bits):
    if backend == "nvfp4":
        return O.nvfp4_quantize_ref(w_bits)
    if backend == "mxfp4":
        return O.mxfp4_quantize_ref(w_bits)
    return O.bf16_bits_to_f32(w_bits).astype(np.float64)


def linear(backend, x, wq, bias_bits):
    """BF16 output of one linear on BF16-valued float64 input x."""
    xb = bits(x)
    if backend == "nvfp4":
        out, _ = O.nvfp4_linear_ref(xb, *wq, bias_bits)
    elif backend == "mxfp4":
        out, _ = O.mxfp4_linear_ref(xb, *wq, bias_bits)
    else:
        out = O.bf16_bits_to_f32(xb).astype(np.float64) @ wq.T
        out = out + O.bf16_bits_to_f32(bias_bits).astype(np.float64)[None, :]
    return bf16_round(out)


def rmsnorm(x):
    return bf16_round(x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + EPS))


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def attention(qkv, rollouts, tokens, heads, hd):
    q, k, v = (qkv.reshape(rollouts, tokens, 3, heads, hd)[:, :, i].transpose(0, 2, 1, 3)
               for i in range(3))
    s = q @ k.transpose(0, 1, 3, 2) / np.sqrt(hd)
    s = np.exp(s - s.max(axis=-1, keepdims=True))
    p = s / s.sum(axis=-1, keepdims=True)
    a = (p @ v).transpose(0, 2, 1, 3).reshape(rollouts * tokens, heads * hd)
    return bf16_round(a)


def blocks(backend, x, layers, cfg):
    for L in layers:
        h = rmsnorm(x)
        qkv = linear(backend, h, *L["qkv"])
        a = attention(qkv, cfg.rollouts, cfg.tokens, cfg.heads, cfg.hidden // cfg.heads)
        x = bf16_round(x + linear(backend, a, *L["out"]))
        h = rmsnorm(x)
        u = bf16_round(gelu_tanh(linear(backend, h, *L["up"])))
        x = bf16_round(x + linear(backend, u, *L["down"]))
    return x


def rollout(backend, x0_bits, weights, cfg):
    """weights: per block {name: (w_bits, bias_bits)}; returns the final
    latents (float64, BF16-valued)."""
    layers = [{n: (prepare(backend, w), b) for n, (w, b) in blk.items()} for blk in weights]
    x = O.bf16_bits_to_f32(x0_bits).astype(np.float64)
    dt = 1.0 / cfg.steps
    for _ in range(cfg.steps):
        y = blocks(backend, x, layers, cfg)
        x = bf16_round(x + dt * (y - x))
    return x


def rewards(x_final, u, cfg):
    return (x_final.reshape(cfg.rollouts, cfg.tokens, cfg.hidden) @ u.astype(np.float64)).mean(axis=1)
