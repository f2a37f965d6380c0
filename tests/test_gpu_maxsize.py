"""GPU parity at sizes past 32-bit byte offsets: both quantizers on a tensor
of more than 2^31 BF16 elements (over 4 GiB), and both GEMMs with an
output of more than 4 GiB.  The whole tensors are far beyond what the CPU
oracle can take, so the check runs on sampled rows: the first and last rows
and the rows on both sides of every 4 GiB boundary of each buffer.  Codes,
scales and alpha must be bit-identical; GEMM rows meet the per-element bound
and the 2e-3 relative Frobenius bound against the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle.nvfp4 as O
import paper_2604_06916_amd as sol
from gpu_util import (abs_products, assert_per_element, bf16_from_dev, device, f32_bits,
                      poison_bf16, poison_u8, rel_fro, say, u8_from_dev)

pytestmark = pytest.mark.gpu

GIB4 = 1 << 32


def boundary_rows(rows, *row_bytes):
    """The first two and last two rows, and the rows on both sides of every
    multiple of 4 GiB in buffers of `row_bytes` bytes per row."""
    out = {0, 1, rows - 2, rows - 1}
    for rb in row_bytes:
        b = GIB4
        while b < rows * rb:
            r = b // rb
            out |= {r - 1, r, r + 1}
            b += GIB4
    return sorted(r for r in out if 0 <= r < rows)


def seeded(seed):
    g = torch.Generator(device=device())
    g.manual_seed(seed)
    return g


def bits_rows(t, rows):
    return t[torch.tensor(rows, device=t.device)].view(torch.int16).cpu().numpy().view(np.uint16)


def test_quantize_past_4gib():
    rows, K = (1 << 20) + 5, 2080          # 2.18e9 elements, 4.4 GB of BF16, 130 blocks of 16 per row
    x = torch.randn((rows, K), dtype=torch.float32, device=device(), generator=seeded(11))
    x = x.to(torch.bfloat16)
    planted = rows - 3
    x[planted, 17] = 100.0                 # the tensor's largest magnitude, so alpha is known
    codes = poison_u8((rows, K // 2))
    scales = poison_u8((rows, K // 16))
    gs = torch.full((1,), float("nan"), dtype=torch.float32, device=device())
    say(f"  quantize {rows} x {K} ({rows * K * 2 / 2**30:.2f} GiB)")
    sol.nvfp4_quantize(x, codes, scales, gs)
    torch.cuda.synchronize()
    sample = sorted(set(boundary_rows(rows, 2 * K, K // 2, K // 16)) | {planted})
    xb = bits_rows(x, sample)
    rc, rs, ra = O.nvfp4_quantize_ref(xb)
    a = np.float32(gs.cpu().numpy()[0])
    assert f32_bits(a) == f32_bits(ra), (a, ra)
    idx = torch.tensor(sample, device=device())
    assert np.array_equal(u8_from_dev(scales[idx]), rs)
    assert np.array_equal(u8_from_dev(codes[idx]), rc)
    say(f"  {len(sample)} sampled rows bit-exact, alpha {a!r}")
    del codes, scales
    # the MXFP4 quantize on the same tensor (its blocks are independent)
    mcodes = poison_u8((rows, K // 2))
    mscales = poison_u8((rows, K // 32))
    sol.mxfp4_quantize(x, mcodes, mscales)
    torch.cuda.synchronize()
    mc, ms = O.mxfp4_quantize_ref(xb)
    assert np.array_equal(u8_from_dev(mscales[idx]), ms)
    assert np.array_equal(u8_from_dev(mcodes[idx]), mc)
    say(f"  MXFP4: {len(sample)} sampled rows bit-exact")
    del x, mcodes, mscales
    torch.cuda.empty_cache()


@pytest.mark.parametrize("fmt", ["nvfp4", "mxfp4"])
def test_gemm_output_past_4gib(fmt):
    M, N, K = (1 << 21) + 40, 1024, 256    # output 4.3 GB; rows 2^21 - 1 .. 2^21 + 1 straddle 4 GiB
    blk = 16 if fmt == "nvfp4" else 32
    g = seeded(12)
    ac = torch.randint(0, 256, (M, K // 2), dtype=torch.uint8, device=device(), generator=g)
    bc = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device=device(), generator=g)
    if fmt == "nvfp4":      # E4M3 scales 0.5 .. 1.75
        lo, hi = 0x30, 0x3F
    else:                   # E8M0 scales 2^-4 .. 2^3
        lo, hi = 123, 131
    as_ = torch.randint(lo, hi, (M, K // blk), dtype=torch.uint8, device=device(), generator=g)
    bs = torch.randint(lo, hi, (N, K // blk), dtype=torch.uint8, device=device(), generator=g)
    rng = np.random.default_rng(13)
    bias_bits = O.f64_to_bf16_bits_rne(rng.normal(0.0, 0.5, N))
    bias = torch.from_numpy(bias_bits.view(np.int16)).to(device()).view(torch.bfloat16)
    out = poison_bf16((M, N))
    say(f"  {fmt} GEMM {M} x {N} x {K} (output {M * N * 2 / 2**30:.2f} GiB)")
    if fmt == "nvfp4":
        ag = torch.tensor([0.5], dtype=torch.float32, device=device())
        bg = torch.tensor([0.25], dtype=torch.float32, device=device())
        sol.nvfp4_gemm(ac, as_, ag, bc, bs, bg, bias, out)
    else:
        sol.mxfp4_gemm(ac, as_, bc, bs, bias, out)
    torch.cuda.synchronize()
    rows = boundary_rows(M, 2 * N)
    assert (1 << 21) in rows
    idx = torch.tensor(rows, device=device())
    a_c, a_s = u8_from_dev(ac[idx]), u8_from_dev(as_[idx])
    b_c, b_s = u8_from_dev(bc), u8_from_dev(bs)
    got = bf16_from_dev(out[idx])
    if fmt == "nvfp4":
        ref = O.nvfp4_gemm_ref(a_c, a_s, 0.5, b_c, b_s, 0.25, bias_bits)
        sabs = abs_products(O.nvfp4_unscaled_ref(a_c, a_s), O.nvfp4_unscaled_ref(b_c, b_s))
        alpha = 0.125
    else:
        ref = O.mxfp4_gemm_ref(a_c, a_s, b_c, b_s, bias_bits)
        sabs = abs_products(O.mxfp4_unscaled_ref(a_c, a_s), O.mxfp4_unscaled_ref(b_c, b_s))
        alpha = 1.0
    err = rel_fro(got, ref)
    say(f"  {len(rows)} sampled rows: rel_fro {err:.3e}")
    assert err <= 2e-3
    assert_per_element(got, ref, sabs, alpha, K, bias_bits, label=f"{fmt} ")
    del ac, bc, as_, bs, out
    torch.cuda.empty_cache()
