"""nvfp4_linear on the GPU: bit-identical to nvfp4_quantize followed by
nvfp4_gemm, and within tolerance of the oracle's quantize-then-GEMM."""
import numpy as np
import pytest
import torch

import oracle.nvfp4 as O
import paper_2604_06916_amd as sol
from gpu_util import (abs_products, assert_per_element, bf16_from_dev, bf16_mismatch_fraction,
                      bf16_to_dev, poison_bf16, rel_fro, say)
from workloads import draw_activations, draw_bias, draw_weights

pytestmark = pytest.mark.gpu


# 4352 x 4096 x 1536 and 128 x 3072 x 3072: the GEMM's last round splits into
# K halves (256 x 256 and 128 x 128 tiles), through the part of the linear's
# workspace after the activation codes
# Few tokens with K % 128 == 0 take a few-token GEMM: the wave-K kernel
# (128 x 1152 x 1152, 128 x 3072 x 3072, ragged 100 x 200 x 384, 65 x 130 x
# 256 with N % 8 != 0, 1 x 16 x 128) or the 64 x 64 one (256 x 1152 x 1152,
# 300 x 1000 x 512, 320 x 1024 x 256); where the latter runs with K <= 512
# (the last two), nvfp4_linear quantizes the activations inside it: still
# bit-identical to nvfp4_quantize followed by nvfp4_gemm
@pytest.mark.parametrize("M,N,K", [(1, 16, 16), (7, 33, 48), (128, 1152, 1152), (300, 520, 2240),
                                   (517, 260, 5600), (1000, 3072, 3072), (4352, 4096, 1536),
                                   (128, 3072, 3072), (100, 200, 384), (65, 130, 256), (1, 16, 128),
                                   (256, 1152, 1152), (300, 1000, 512), (320, 1024, 256)])
@pytest.mark.parametrize("with_bias", [False, True])
def test_linear_matches_quantize_then_gemm_and_oracle(M, N, K, with_bias):
    xb = draw_activations("t3_1pct", M, K, seed=M + K)
    wb = draw_weights(N, K, 0.02, seed=N + K)
    bias = draw_bias(N, 0.02, seed=N) if with_bias else None
    x, w = bf16_to_dev(xb), bf16_to_dev(wb)
    b = None if bias is None else bf16_to_dev(bias)
    wc, ws, wa = sol.nvfp4_quantize(w)
    out = poison_bf16((M, N))
    sol.nvfp4_linear(x, wc, ws, wa, b, out)
    xc, xs, xa = sol.nvfp4_quantize(x)
    out2 = sol.nvfp4_gemm(xc, xs, xa, wc, ws, wa, b)
    torch.cuda.synchronize()
    got = bf16_from_dev(out)
    assert np.array_equal(got, bf16_from_dev(out2))

    rw = O.nvfp4_quantize_ref(wb)
    ref, rx = O.nvfp4_linear_ref(xb, *rw, bias)
    err = rel_fro(got, ref)
    mism = bf16_mismatch_fraction(got, ref)
    say(f"linear M={M} N={N} K={K} bias={with_bias}: rel_fro={err:.3e} mismatch={mism:.2e}")
    assert err <= 2e-3
    assert mism <= 0.01
    sabs = abs_products(O.nvfp4_unscaled_ref(rx[0], rx[1]), O.nvfp4_unscaled_ref(rw[0], rw[1]))
    assert_per_element(got, ref, sabs, np.float32(rx[2]) * np.float32(rw[2]), K, bias)


def test_linear_workspace_holds_the_activation_codes():
    M, N, K = 64, 48, 256
    xb = draw_activations("normal", M, K, seed=3)
    wb = draw_weights(N, K, 0.02, seed=4)
    x = bf16_to_dev(xb)
    wc, ws, wa = sol.nvfp4_quantize(bf16_to_dev(wb))
    wsp = torch.empty(sol.nvfp4_linear_workspace_bytes(M, N, K), dtype=torch.uint8, device=x.device)
    sol.nvfp4_linear(x, wc, ws, wa, workspace=wsp)
    torch.cuda.synchronize()
    rc, _, _ = O.nvfp4_quantize_ref(xb)
    assert np.array_equal(wsp[: M * K // 2].cpu().numpy().reshape(M, K // 2), rc)


@pytest.mark.parametrize("M,N,K", [(64, 48, 256), (100, 200, 384), (300, 1000, 512),
                                   (320, 1024, 256), (128, 1152, 1152)])
def test_fused_linear_leaves_codes_scales_and_alpha(M, N, K):
    """Every small-token route (the fused one, 300 x 1000 x 512 and
    320 x 1024 x 256; amax + encode + a few-token GEMM otherwise) leaves the
    activations' codes, scales and alpha in the workspace exactly as
    nvfp4_quantize would (codes at offset 0, then the scales and alpha, each
    region 256-byte aligned)."""
    import paper_2604_06916_amd as sol2
    assert sol2.gemm_plan(M, N, K)["kernel"] in ("nvfp4_gemm_small_kernel", "nvfp4_gemm_wavek_kernel")
    xb = draw_activations("outlier4x20", M, K, seed=M + 5)
    wb = draw_weights(N, K, 0.02, seed=N + 6)
    x = bf16_to_dev(xb)
    wc, ws, wa = sol.nvfp4_quantize(bf16_to_dev(wb))
    wsp = torch.full((sol.nvfp4_linear_workspace_bytes(M, N, K),), 0xAB, dtype=torch.uint8,
                     device=x.device)
    sol.nvfp4_linear(x, wc, ws, wa, workspace=wsp)
    torch.cuda.synchronize()
    rc, rs, ra = O.nvfp4_quantize_ref(xb)
    buf = wsp.cpu().numpy()
    assert np.array_equal(buf[: M * K // 2].reshape(M, K // 2), rc)
    soff = (M * K // 2 + 255) // 256 * 256
    assert np.array_equal(buf[soff: soff + M * K // 16].reshape(M, K // 16), rs)
    aoff = soff + (M * K // 16 + 255) // 256 * 256
    assert buf[aoff: aoff + 4].view(np.float32)[0] == ra


def test_fused_linear_zero_and_signed_zero_input():
    """All-zero activations (alpha = 0, every scale 0, codes keep the sign
    of zero) through the fused path (320 x 1024 x 256: the GEMM itself runs
    on 64 x 64 tiles there): the output is the bias, and the codes in the
    workspace are the oracle's."""
    M, N, K = 320, 1024, 256
    xb = np.zeros((M, K), np.uint16)
    xb[::3, ::5] = 0x8000
    wb = draw_weights(N, K, 0.02, seed=9)
    bias = draw_bias(N, 0.02, seed=10)
    x = bf16_to_dev(xb)
    wc, ws, wa = sol.nvfp4_quantize(bf16_to_dev(wb))
    wsp = torch.empty(sol.nvfp4_linear_workspace_bytes(M, N, K), dtype=torch.uint8, device=x.device)
    out = sol.nvfp4_linear(x, wc, ws, wa, bf16_to_dev(bias), workspace=wsp)
    torch.cuda.synchronize()
    assert np.array_equal(bf16_from_dev(out), np.broadcast_to(bias, (M, N)))
    rc, _, _ = O.nvfp4_quantize_ref(xb)
    assert np.array_equal(wsp[: M * K // 2].cpu().numpy().reshape(M, K // 2), rc)
