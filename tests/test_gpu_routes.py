"""Seeded random shapes across every GEMM route (tests/route_shapes.py; the
CPU test test_routes_host.py checks that they meet every kernel, tile size
and the split last round): nvfp4_gemm and mxfp4_gemm against the oracle
(2e-3 relative Frobenius and the per-element FP32 summation bound), and
nvfp4_linear bit-identical to nvfp4_quantize followed by nvfp4_gemm."""
import numpy as np
import pytest
import torch

import oracle.nvfp4 as O
import paper_2604_06916_amd as sol
from gpu_util import (abs_products, assert_per_element, bf16_from_dev, bf16_to_dev, f32_to_dev,
                      poison_bf16, rel_fro, say, u8_to_dev)
from route_shapes import SHAPES
from workloads import draw_activations, draw_bias, draw_weights

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_nvfp4_route_vs_oracle_and_linear(M, N, K):
    plan = sol.gemm_plan(M, N, K)
    xb = draw_activations("t3_1pct", M, K, seed=3 * M + K)
    wb = draw_weights(N, K, 0.02, seed=5 * N + K)
    bias = draw_bias(N, 0.02, seed=N + 7)
    a, b = O.nvfp4_quantize_ref(xb), O.nvfp4_quantize_ref(wb)
    out = poison_bf16((M, N))
    sol.nvfp4_gemm(u8_to_dev(a[0]), u8_to_dev(a[1]), f32_to_dev(a[2]), u8_to_dev(b[0]),
                   u8_to_dev(b[1]), f32_to_dev(b[2]), bf16_to_dev(bias), out)
    torch.cuda.synchronize()
    got = bf16_from_dev(out)
    ref = O.nvfp4_gemm_ref(*a, *b, bias)
    err = rel_fro(got, ref)
    say(f"{M}x{N}x{K} {plan['kernel']} tile {plan['tile']} splits {plan['splits']}: rel_fro {err:.3e}")
    assert err <= 2e-3
    sabs = abs_products(O.nvfp4_unscaled_ref(a[0], a[1]), O.nvfp4_unscaled_ref(b[0], b[1]))
    assert_per_element(got, ref, sabs, np.float32(a[2]) * np.float32(b[2]), K, bias)
    # the linear on the same layer, from BF16: identical to quantize + gemm
    x, w, bd = bf16_to_dev(xb), bf16_to_dev(wb), bf16_to_dev(bias)
    wc, ws, wa = sol.nvfp4_quantize(w)
    lin = sol.nvfp4_linear(x, wc, ws, wa, bd)
    xc, xs, xa = sol.nvfp4_quantize(x)
    two = sol.nvfp4_gemm(xc, xs, xa, wc, ws, wa, bd)
    torch.cuda.synchronize()
    assert np.array_equal(bf16_from_dev(lin), bf16_from_dev(two))


@pytest.mark.parametrize("M,N,K", [(M, N, K - K % 32) for M, N, K in SHAPES if K >= 32])
def test_mxfp4_route_vs_oracle(M, N, K):
    plan = sol.gemm_plan(M, N, K, sol.FORMAT_MXFP4)
    ac, as_ = O.mxfp4_quantize_ref(draw_activations("normal", M, K, seed=7 * M + K))
    bc, bs = O.mxfp4_quantize_ref(draw_weights(N, K, 0.02, seed=11 * N + K))
    bias = draw_bias(N, 0.02, seed=N + 9)
    out = poison_bf16((M, N))
    sol.mxfp4_gemm(u8_to_dev(ac), u8_to_dev(as_), u8_to_dev(bc), u8_to_dev(bs), bf16_to_dev(bias), out)
    torch.cuda.synchronize()
    got = bf16_from_dev(out)
    ref = O.mxfp4_gemm_ref(ac, as_, bc, bs, bias)
    err = rel_fro(got, ref)
    say(f"MXFP4 {M}x{N}x{K} tile {plan['tile']}: rel_fro {err:.3e}")
    assert err <= 2e-3
    sabs = abs_products(O.mxfp4_unscaled_ref(ac, as_), O.mxfp4_unscaled_ref(bc, bs))
    assert_per_element(got, ref, sabs, 1.0, K, bias)
