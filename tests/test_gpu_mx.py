"""GPU parity of the MXFP4 path (mxfp4_quantize, mxfp4_gemm, mxfp4_linear)
against the CPU oracle.

Quantization is an encoding with exactly one correct result, so codes and
E8M0 scales must be bit-identical.  GEMM operands are quantized by the oracle
and uploaded, so the GEMM is tested on the oracle's own inputs: bit-exact
where every FP32 sum is exact, else relative Frobenius error <= 2e-3 against
the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle.nvfp4 as O
import paper_2604_06916_amd as sol
from gpu_util import (abs_products, assert_per_element, bf16_from_dev, bf16_mismatch_fraction,
                      bf16_to_dev, device, poison_bf16,
                      poison_u8, rel_fro, say, u8_from_dev, u8_to_dev)
from workloads import draw_activations, draw_bias, draw_weights, f32_to_bf16_bits

pytestmark = pytest.mark.gpu

TOL = 2e-3
KINDS = ["normal", "outlier4x20", "t3_1pct", "gelu", "rowscale", "uniform"]


def gpu_quant(xb):
    rows, K = xb.shape
    codes, scales = poison_u8((rows, K // 2)), poison_u8((rows, K // 32))
    sol.mxfp4_quantize(bf16_to_dev(xb), codes, scales)
    torch.cuda.synchronize()
    return u8_from_dev(codes), u8_from_dev(scales)


def assert_quant_matches(xb, label=""):
    c, s = gpu_quant(xb)
    rc, rs = O.mxfp4_quantize_ref(xb)
    if not np.array_equal(s, rs):
        r, b = np.argwhere(s != rs)[0]
        raise AssertionError(f"{label}: scale [{r},{b}] gpu {s[r, b]:#x} oracle {rs[r, b]:#x}")
    if not np.array_equal(c, rc):
        r, j = np.argwhere(c != rc)[0]
        raise AssertionError(f"{label}: code byte [{r},{j}] gpu {c[r, j]:#x} oracle {rc[r, j]:#x}")


def gpu_gemm(ac, as_, bc, bs, bias=None):
    M, N = ac.shape[0], bc.shape[0]
    out = poison_bf16((M, N))
    sol.mxfp4_gemm(u8_to_dev(ac), u8_to_dev(as_), u8_to_dev(bc), u8_to_dev(bs),
                   None if bias is None else bf16_to_dev(bias), out)
    torch.cuda.synchronize()
    return bf16_from_dev(out)


# ---------------------------------------------------------------- quantize

def test_golden_quantize():
    import golden_io
    for name, c in golden_io.load().items():
        if c["kind"] != "mxcase":
            continue
        xb = f32_to_bf16_bits(np.asarray(c["x"], dtype=np.float32))[None, :]
        codes, scales = gpu_quant(xb)
        assert codes.tobytes() == c["codes"].tobytes(), name
        assert scales.tobytes() == c["mxscales"].tobytes(), name


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("rows,K", [(1, 32), (3, 96), (37, 1152), (300, 2240), (129, 5600)])
def test_quantize_random(kind, rows, K):
    xb = draw_activations(kind, rows, K, rows * 7 + K)
    assert_quant_matches(xb, f"{kind} {rows}x{K}")


def test_quantize_every_bf16_pattern():
    """Every finite BF16 bit pattern appears as an element of a block whose
    other elements lie in the same binade (patterns sorted by magnitude), with
    the block amax raised by 0-5 binades, so each pattern lands on every part
    of the E2M1 range across all scale bytes (subnormal and zero amax
    included)."""
    pats = np.arange(0x10000, dtype=np.uint32)
    pats = pats[((pats >> 7) & 0xFF) != 0xFF].astype(np.uint16)
    pats = pats[np.argsort(pats & 0x7FFF, kind="stable")]
    g = np.random.Generator(np.random.PCG64(5))
    n = pats.size // 31 * 31
    body = pats[:n].reshape(-1, 31)
    mag = (body & 0x7FFF).max(axis=1).astype(np.uint32)
    bump = np.minimum(mag + (g.integers(0, 6, size=mag.size) << 7), 0x7F7F).astype(np.uint16)
    blocks = np.concatenate([body, bump[:, None]], axis=1)
    xb = blocks[: blocks.shape[0] // 8 * 8].reshape(-1, 32 * 8)
    _, rs = O.mxfp4_quantize_ref(xb)
    assert rs.min() == 0 and rs.max() >= 252
    assert_quant_matches(xb, "all patterns")


def test_quantize_ties_and_saturation():
    """Elements on every E2M1 midpoint and beyond 6 at many scales: ties go to
    the even code, magnitudes in (6, 8) saturate."""
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.5, 7.0, 7.5, 7.875, 6.0, 0.0],
                    dtype=np.float32)
    rows = []
    for e in range(-120, 120, 7):
        blk = np.zeros(32, np.float32)
        blk[: mids.size] = mids * np.float32(2.0 ** e)
        blk[mids.size: 2 * mids.size] = -mids * np.float32(2.0 ** e)
        rows.append(blk)
    xb = f32_to_bf16_bits(np.stack(rows))
    assert_quant_matches(xb, "ties")


def test_quantize_zero_blocks_and_signed_zeros():
    xb = np.zeros((4, 128), np.uint16)
    xb[1, 5] = 0x8000
    xb[2, 40:72] = 0x8000
    xb[3, 100] = 0x0001          # smallest subnormal
    assert_quant_matches(xb, "zeros")


@pytest.mark.parametrize("nblocks", [1, 3, 4, 5, 511, 513, 1027])
def test_quantize_block_counts(nblocks):
    """Tails of the 4-block scale stores."""
    xb = draw_activations("normal", nblocks, 32, nblocks)
    assert_quant_matches(xb, f"{nblocks} blocks")


def test_quantize_grid_stride():
    """More blocks than one sweep of the capped grid covers (8192 workgroups
    x 512 blocks), with a ragged tail.  MX blocks are encoded independently,
    so the expected result of a tiled input is the tiled oracle result."""
    base = draw_activations("t3_1pct", 4099, 32, 9)
    reps = (8192 * 512 + 77 + base.shape[0] - 1) // base.shape[0]
    nblocks = 8192 * 512 + 77
    xb = np.tile(base, (reps, 1))[:nblocks]
    rc, rs = O.mxfp4_quantize_ref(base)
    c, s = gpu_quant(xb)
    assert np.array_equal(s, np.tile(rs, (reps, 1))[:nblocks])
    assert np.array_equal(c, np.tile(rc, (reps, 1))[:nblocks])


def test_quantize_empty():
    x = torch.empty((0, 64), dtype=torch.bfloat16, device=device())
    c, s = sol.mxfp4_quantize(x)
    torch.cuda.synchronize()
    assert c.shape == (0, 32) and s.shape == (0, 2)


# -------------------------------------------------------------------- GEMM

def test_golden_gemm():
    import golden_io
    for name, c in golden_io.load().items():
        if c["kind"] != "mxgemm":
            continue
        got = gpu_gemm(c["a_codes"][None], c["a_scales"][None], c["b_codes"][None],
                       c["b_scales"][None])
        assert int(got[0, 0]) == c["bf16"], name


# The small shapes run on 64 x 64 tiles or, where K spans several 128-element
# stages ((64, 96, 512), (260, 300, 1152)), on the wave-K kernel; (1000, 3000,
# K) and (1024, 3072, K) on 128 x 128 tiles, (4200, 4360, K) and (6000, 6152,
# 1024) on 256 x 256 ones (ragged M and N); (4353, 4100, 96) and (4224, 4001,
# 1024) on 256 x 256 tiles whose last round (50 and 16 tiles) runs as 128 x 128
# quadrants in a second launch, some of them outside the output.  Scale groups (16 bytes of a row) are one 16-byte load;
# with K % 128 != 0 (K = 96, 2240) rows start at any byte offset and the lane
# of an operand's last row whose group reaches past the range loads bytes
# instead, on every tile size.  K = 1152 (K % 512 !=
# 0) once fetched groups as four 4-byte loads that the compiler merged (a
# stage-end wait that counted them as four let the previous stage's loads
# still be in flight).
@pytest.mark.parametrize("M,N,K", [(1, 1, 32), (3, 5, 64), (37, 70, 128), (300, 260, 96),
                                   (257, 513, 32), (64, 96, 512), (260, 300, 1152),
                                   (1000, 3000, 128), (1024, 3072, 96),
                                   (4200, 4360, 1024), (6000, 6152, 1024), (4200, 4360, 1152),
                                   (300, 260, 2240), (4200, 4360, 2240), (4201, 4359, 96),
                                   (4353, 4100, 96), (4224, 4001, 1024)])
def test_exact_sums_are_bit_exact(M, N, K):
    """Scales 2^-2 and 2^3: every partial sum is a multiple of 1/2 below
    2^17, exact in FP32, so the only rounding is the final BF16."""
    g = np.random.Generator(np.random.PCG64(M * 1000 + N + K))
    ac = g.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
    bc = g.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    as_ = np.full((M, K // 32), 125, np.uint8)
    bs = np.full((N, K // 32), 130, np.uint8)
    ref = O.mxfp4_gemm_ref(ac, as_, bc, bs)
    got = gpu_gemm(ac, as_, bc, bs)
    assert np.array_equal(got, O.bf16_output(ref))


def one_hot(n, K):
    h4 = np.zeros((n, K), np.uint8)
    h4[np.arange(n), np.arange(n)] = 0x2
    return O.pack_codes(h4), np.full((n, K // 32), 127, np.uint8)


@pytest.mark.parametrize("side", ["A", "B"])
def test_every_scale_code_bit_exact(side):
    """One operand cycles its scales through the E8M0 codes 2..252 (every
    decoded value a normal FP32 and BF16 number) with random codes; the other
    is one-hot (value 1 at k = row).  Each output is one exact product, so it
    equals the decoded element exactly; pins the per-lane scale selection,
    nibble order and both operand sides."""
    R, K = 300, 288
    g = np.random.Generator(np.random.PCG64(51 if side == "A" else 52))
    c = g.integers(0, 256, size=(R, K // 2), dtype=np.uint8)
    sc = (2 + np.arange(R * (K // 32)).reshape(R, K // 32) % 251).astype(np.uint8)
    hc, hs = one_hot(260, K)
    args = (c, sc, hc, hs) if side == "A" else (hc, hs, c, sc)
    ref = O.mxfp4_gemm_ref(*args)
    got = gpu_gemm(*args)
    assert np.array_equal(got, O.bf16_output(ref))


SHAPES = [(1, 1, 32), (5, 7, 64), (64, 64, 128), (255, 257, 96), (300, 520, 288),
          (257, 129, 2240), (128, 1152, 1152), (513, 260, 5600), (96, 300, 3072),
          (260, 2049, 256), (600, 700, 2432),
          # 128 x 128 tiles (the shapes above take 64 x 64 ones)
          (1000, 3000, 256), (1024, 3072, 160),
          # 256 x 256 tiles, more tiles than compute units
          (4200, 4360, 1024), (2100, 9000, 3072),
          # ... and a last round of 16 or 50 tiles as 128 x 128 quadrants
          (4224, 4001, 1024), (4353, 4100, 2240)]


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("with_bias", [False, True])
def test_random_vs_oracle(M, N, K, with_bias):
    ac, as_ = O.mxfp4_quantize_ref(draw_activations("normal", M, K, 7 * M + K))
    bc, bs = O.mxfp4_quantize_ref(draw_weights(N, K, 0.02, 11 * N + K))
    bias = draw_bias(N, 0.02, N) if with_bias else None
    ref = O.mxfp4_gemm_ref(ac, as_, bc, bs, bias)
    got = gpu_gemm(ac, as_, bc, bs, bias)
    err = rel_fro(got, ref)
    mism = bf16_mismatch_fraction(got, ref)
    floor = rel_fro(O.bf16_output(ref), ref)
    say(f"M={M} N={N} K={K} bias={with_bias}: rel_fro={err:.3e} (bf16 floor {floor:.3e}) "
        f"mismatch={mism:.2e}")
    assert np.isfinite(O.bf16_bits_to_f32(got)).all()
    assert err <= TOL
    assert mism <= 0.01
    sabs = abs_products(O.mxfp4_unscaled_ref(ac, as_), O.mxfp4_unscaled_ref(bc, bs))
    assert_per_element(got, ref, sabs, 1.0, K, bias)


# Few tokens on the wave-K kernel (32 x 32 tiles, each workgroup's K stages
# dealt to its four waves, their sums added in LDS in wave order): 2 stages
# (two waves without one), 3, 5 (uneven shares), 9 and 36 stages; ragged M
# and N, N % 8 != 0.
MX_WAVEK_SHAPES = [(7, 33, 256), (100, 200, 384), (33, 40, 640), (65, 130, 1152),
                   (128, 1152, 1152), (128, 1152, 4608)]


@pytest.mark.parametrize("M,N,K", MX_WAVEK_SHAPES)
def test_wavek_kernel_vs_oracle(M, N, K):
    assert sol.gemm_plan(M, N, K, sol.FORMAT_MXFP4)["kernel"] == "mxfp4_gemm_wavek_kernel"
    ac, as_ = O.mxfp4_quantize_ref(draw_activations("outlier4x20", M, K, 31 * M + K))
    bc, bs = O.mxfp4_quantize_ref(draw_weights(N, K, 0.02, 37 * N + K))
    bias = draw_bias(N, 0.02, N + 3)
    got = gpu_gemm(ac, as_, bc, bs, bias)
    assert np.array_equal(got, gpu_gemm(ac, as_, bc, bs, bias))   # fixed sum order
    ref = O.mxfp4_gemm_ref(ac, as_, bc, bs, bias)
    err = rel_fro(got, ref)
    say(f"wave-K M={M} N={N} K={K}: rel_fro={err:.3e}")
    assert err <= TOL
    assert bf16_mismatch_fraction(got, ref) <= 0.01
    sabs = abs_products(O.mxfp4_unscaled_ref(ac, as_), O.mxfp4_unscaled_ref(bc, bs))
    assert_per_element(got, ref, sabs, 1.0, K, bias)


@pytest.mark.parametrize("M,N,K", [(7, 33, 256), (33, 40, 640), (128, 1152, 4608)])
def test_wavek_exact_sums_are_bit_exact(M, N, K):
    """As test_exact_sums_are_bit_exact, on the wave-K kernel: the sum of
    the four waves' partial sums is exact too."""
    assert sol.gemm_plan(M, N, K, sol.FORMAT_MXFP4)["kernel"] == "mxfp4_gemm_wavek_kernel"
    g = np.random.Generator(np.random.PCG64(M * 1000 + N + K + 7))
    ac = g.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
    bc = g.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    as_ = np.full((M, K // 32), 125, np.uint8)
    bs = np.full((N, K // 32), 130, np.uint8)
    ref = O.mxfp4_gemm_ref(ac, as_, bc, bs)
    got = gpu_gemm(ac, as_, bc, bs)
    assert np.array_equal(got, O.bf16_output(ref))


def test_quadrant_plans():
    """The last round's 256 x 256 tiles as quadrants: 4 workgroups each in
    a second launch (the plan counts both launches)."""
    for M, N in [(4224, 4001), (4353, 4100), (18432, 9216)]:
        tiles = ((M + 255) // 256) * ((N + 255) // 256)
        rem = tiles % 256
        assert 0 < rem <= 64
        p = sol.gemm_plan(M, N, 1024, sol.FORMAT_MXFP4)
        assert p == {"kernel": "mxfp4_gemm_kernel", "tile": 256, "workgroups": tiles + 3 * rem,
                     "splits": 1}


def test_wide_dynamic_range_vs_oracle():
    g = np.random.Generator(np.random.PCG64(61))
    M, N, K = 300, 260, 1024

    def draw(rows):
        x = g.standard_normal((rows, K)).astype(np.float32)
        x *= np.repeat(np.exp2(g.integers(-30, 30, size=(rows, K // 32))), 32, axis=1).astype(np.float32)
        return O.mxfp4_quantize_ref(f32_to_bf16_bits(x))
    a, b = draw(M), draw(N)
    ref = O.mxfp4_gemm_ref(*a, *b)
    got = gpu_gemm(*a, *b)
    err = rel_fro(got, ref)
    say(f"wide: rel_fro={err:.3e}")
    assert err <= TOL
    sabs = abs_products(O.mxfp4_unscaled_ref(*a), O.mxfp4_unscaled_ref(*b))
    assert_per_element(got, ref, sabs, 1.0, K)


def test_zero_k_writes_bias():
    M, N = 33, 70
    bias = draw_bias(N, 0.5, 1)
    out = poison_bf16((M, N))
    z = torch.empty((M, 0), dtype=torch.uint8, device=device())
    zb = torch.empty((N, 0), dtype=torch.uint8, device=device())
    sol.mxfp4_gemm(z, z, zb, zb, bf16_to_dev(bias), out)
    torch.cuda.synchronize()
    assert np.array_equal(bf16_from_dev(out), np.broadcast_to(bias, (M, N)))


def test_gemm_deterministic():
    M, N, K = 1000, 1500, 3072
    ac, as_ = O.mxfp4_quantize_ref(draw_activations("normal", M, K, 1))
    bc, bs = O.mxfp4_quantize_ref(draw_weights(N, K, 0.015, 2))
    assert np.array_equal(gpu_gemm(ac, as_, bc, bs), gpu_gemm(ac, as_, bc, bs))


# ------------------------------------------------------------------ linear

@pytest.mark.parametrize("M,N,K", [(1, 64, 32), (200, 272, 1152), (513, 300, 2240),
                                   (260, 520, 3072)])
def test_linear_equals_quantize_then_gemm(M, N, K):
    xb = draw_activations("t3_1pct", M, K, M + K)
    wc, ws = O.mxfp4_quantize_ref(draw_weights(N, K, 0.02, N + K))
    bias = draw_bias(N, 0.02, N)
    x, wcd, wsd, bd = bf16_to_dev(xb), u8_to_dev(wc), u8_to_dev(ws), bf16_to_dev(bias)
    ws_bytes = sol.mxfp4_linear_workspace_bytes(M, K)
    work = poison_u8((ws_bytes,))
    out = poison_bf16((M, N))
    sol.mxfp4_linear(x, wcd, wsd, bd, out, work)
    xc, xs = sol.mxfp4_quantize(x)
    out2 = sol.mxfp4_gemm(xc, xs, wcd, wsd, bd)
    torch.cuda.synchronize()
    got = bf16_from_dev(out)
    assert np.array_equal(got, bf16_from_dev(out2))
    rc, rs = O.mxfp4_quantize_ref(xb)
    assert np.array_equal(u8_from_dev(work[: M * K // 2]).reshape(M, K // 2), rc)
    ref, _ = O.mxfp4_linear_ref(xb, wc, ws, bias)
    err = rel_fro(got, ref)
    say(f"linear M={M} N={N} K={K}: rel_fro={err:.3e}")
    assert err <= TOL
    sabs = abs_products(O.mxfp4_unscaled_ref(rc, rs), O.mxfp4_unscaled_ref(wc, ws))
    assert_per_element(got, ref, sabs, 1.0, K, bias)
