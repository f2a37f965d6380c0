"""nvfp4_quantize_noalloc, the allocation-free quantize (its partial maxima
live in the library's fixed per-device scratch array): called through the
C-ABI, its codes, scales and alpha must equal nvfp4_quantize's bit for bit,
on two calls in a row (the second on a smaller input, so stale partials of
the first call sit in the scratch past the ones the second uses), then once
more on the first input."""
import numpy as np
import pytest
import torch

import paper_2604_06916_amd as sol
from gpu_util import bf16_to_dev, device, f32_bits, say, u8_from_dev
from workloads import draw_activations

pytestmark = pytest.mark.gpu


def both(xb):
    x = bf16_to_dev(xb)
    rows, K = xb.shape
    want = sol.nvfp4_quantize(x)
    codes = torch.full((rows, K // 2), 0xAB, dtype=torch.uint8, device=x.device)
    scales = torch.full((rows, K // 16), 0xAB, dtype=torch.uint8, device=x.device)
    gs = torch.full((1,), float("nan"), dtype=torch.float32, device=x.device)
    sol.nvfp4_quantize_noalloc(x, codes, scales, gs)
    torch.cuda.synchronize()
    return want, (codes, scales, gs)


def check(want, got, label):
    assert np.array_equal(u8_from_dev(got[0]), u8_from_dev(want[0])), label
    assert np.array_equal(u8_from_dev(got[1]), u8_from_dev(want[1])), label
    assert f32_bits(got[2].cpu().numpy()[0]) == f32_bits(want[2].cpu().numpy()[0]), label
    say(f"{label}: codes, scales and alpha bit-identical to nvfp4_quantize")


def test_noalloc_matches_quantize_on_consecutive_calls():
    device()
    big = draw_activations("outlier4x20", 4096, 4096, seed=71)      # 256 partial maxima
    small = draw_activations("t3_1pct", 128, 1152, seed=72)          # 3 partial maxima
    check(*both(big), "first call, 4096 x 4096")
    check(*both(small), "second call, 128 x 1152")
    check(*both(big), "third call, 4096 x 4096 again")


def test_noalloc_zero_rows_and_argument_errors():
    dev = device()
    x = torch.empty((0, 64), dtype=torch.bfloat16, device=dev)
    gs = torch.full((1,), 7.0, dtype=torch.float32, device=dev)
    sol.nvfp4_quantize_noalloc(x, torch.empty((0, 32), dtype=torch.uint8, device=dev),
                               torch.empty((0, 4), dtype=torch.uint8, device=dev), gs)
    torch.cuda.synchronize()
    assert gs.item() == 0.0
    rc = sol.lib.nvfp4_quantize_noalloc(None, 4, 24, None, None, None, None)
    assert rc == -2          # K % 16 is checked before any HIP call
