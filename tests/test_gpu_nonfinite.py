"""Non-finite inputs (NaN, +-Inf) on the GPU.

The library leaves the codes of such tensors unspecified but promises that
they never fault.  Every index the kernels derive from data is a scale code:
the NVFP4 encoder's E4M3 rounding sends NaN and values past 448 to 0x7E, so
its per-code table lookup stays in range, and the MXFP4 encoder and both
GEMMs use scale bytes as values only.  These tests run every entry point on
such inputs and check what does hold:
- both quantizers emit finite scale codes only (never E4M3's NaN code 0x7F);
- MXFP4 scales are per block, so every block free of non-finite values is
  encoded exactly as the oracle encodes it;
- the GEMMs and linears on these operands complete."""
import numpy as np
import pytest
import torch

import oracle.nvfp4 as O
import paper_2604_06916_amd as sol
from gpu_util import bf16_to_dev, device, poison_bf16, poison_u8, say, u8_from_dev, u8_to_dev
from workloads import draw_activations, draw_weights

pytestmark = pytest.mark.gpu

NAN, PINF, NINF = 0x7FC0, 0x7F80, 0xFF80


def with_specials(rows, K, kinds, seed):
    xb = draw_activations("normal", rows, K, seed=seed).copy()
    rng = np.random.default_rng(seed)
    where = []
    for v in kinds:
        r, k = int(rng.integers(rows)), int(rng.integers(K))
        xb[r, k] = v
        where.append((r, k))
    return xb, where


@pytest.mark.parametrize("kinds", [[PINF], [NINF, PINF], [NAN], [NAN, PINF, NINF]])
def test_nvfp4_quantize_and_gemm_complete(kinds):
    M, N, K = 96, 80, 512
    xb, where = with_specials(M, K, kinds, seed=len(kinds) + 7)
    say(f"nvfp4 non-finite {[hex(v) for v in kinds]} at {where}")
    x = bf16_to_dev(xb)
    codes, scales = poison_u8((M, K // 2)), poison_u8((M, K // 16))
    gs = torch.zeros(1, dtype=torch.float32, device=device())
    sol.nvfp4_quantize(x, codes, scales, gs)
    torch.cuda.synchronize()
    s = u8_from_dev(scales)
    assert s.max() <= 0x7E, "a scale byte is not a finite E4M3 code"
    assert not np.isfinite(gs.cpu().numpy()[0])

    wc, ws, wa = sol.nvfp4_quantize(bf16_to_dev(draw_weights(N, K, 0.02, seed=3)))
    out = poison_bf16((M, N))
    sol.nvfp4_gemm(codes, scales, gs, wc, ws, wa, None, out)
    out2 = poison_bf16((M, N))
    sol.nvfp4_linear(x, wc, ws, wa, None, out2)
    torch.cuda.synchronize()
    # the linear quantizes x exactly as above, so both are the same call
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16))


@pytest.mark.parametrize("kinds", [[PINF], [NAN], [NAN, PINF, NINF, NAN]])
def test_mxfp4_blocks_stay_local(kinds):
    M, N, K = 64, 96, 256
    xb, where = with_specials(M, K, kinds, seed=len(kinds) + 11)
    say(f"mxfp4 non-finite {[hex(v) for v in kinds]} at {where}")
    codes, scales = poison_u8((M, K // 2)), poison_u8((M, K // 32))
    sol.mxfp4_quantize(bf16_to_dev(xb), codes, scales)
    torch.cuda.synchronize()
    c, s = u8_from_dev(codes), u8_from_dev(scales)

    # the oracle on the same tensor with the touched blocks zeroed: every
    # other block must come out identical
    clean = xb.copy()
    touched = {(r, k // 32) for r, k in where}
    for r, b in touched:
        clean[r, 32 * b:32 * b + 32] = 0
    rc, rs = O.mxfp4_quantize_ref(clean)
    for r in range(M):
        for b in range(K // 32):
            if (r, b) in touched:
                continue
            assert s[r, b] == rs[r, b], f"scale of block ({r}, {b})"
            assert np.array_equal(c[r, 16 * b:16 * b + 16], rc[r, 16 * b:16 * b + 16]), f"codes of block ({r}, {b})"

    wc, ws = sol.mxfp4_quantize(bf16_to_dev(draw_weights(N, K, 0.02, seed=5)))
    out = poison_bf16((M, N))
    sol.mxfp4_gemm(u8_to_dev(c), u8_to_dev(s), wc, ws, None, out)
    out2 = poison_bf16((M, N))
    sol.mxfp4_linear(bf16_to_dev(xb), wc, ws, None, out2)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16))
