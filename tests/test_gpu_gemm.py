"""GPU parity of nvfp4_gemm against the CPU oracle.

Operands are quantized by the oracle on the CPU and uploaded, so the GEMM is
tested on exactly the oracle's inputs.  Bar: relative Frobenius error
<= 2e-3 against the float64 oracle and every element within the FP32
summation bound of gpu_util.assert_per_element; cases whose FP32 sums are
exact must be bit-identical to the oracle's BF16 rounding."""
import numpy as np
import pytest
import torch

import oracle.nvfp4 as O
import paper_2604_06916_amd as sol
from gpu_util import (abs_products, assert_per_element, bf16_from_dev, bf16_mismatch_fraction,
                      bf16_to_dev, device, f32_to_dev, poison_bf16, rel_fro, say, u8_to_dev)
from workloads import draw_activations, draw_bias, draw_weights

pytestmark = pytest.mark.gpu

TOL = 2e-3


def gpu_gemm(ac, as_, aa, bc, bs, ba, bias=None, split=True):
    M, N = ac.shape[0], bc.shape[0]
    out = poison_bf16((M, N))
    sol.nvfp4_gemm(u8_to_dev(ac), u8_to_dev(as_), f32_to_dev(aa), u8_to_dev(bc), u8_to_dev(bs),
                   f32_to_dev(ba), None if bias is None else bf16_to_dev(bias), out, split=split)
    torch.cuda.synchronize()
    return bf16_from_dev(out)


def check_elements(got, a, b, ref, bias=None, label=""):
    """Per-element bound for a GEMM of quantized operands a, b = (codes,
    scales, alpha)."""
    sabs = abs_products(O.nvfp4_unscaled_ref(a[0], a[1]), O.nvfp4_unscaled_ref(b[0], b[1]))
    alpha = np.float32(np.float32(a[2]) * np.float32(b[2]))
    assert_per_element(got, ref, sabs, alpha, a[0].shape[1] * 2, bias, label)


def quantized(kind, rows, K, seed, sigma=None):
    xb = (draw_weights(rows, K, sigma, seed) if sigma is not None
          else draw_activations(kind, rows, K, seed))
    return O.nvfp4_quantize_ref(xb)


def test_golden_gemms():
    import golden_io
    for name, c in golden_io.load().items():
        if c["kind"] != "gemm":
            continue
        got = gpu_gemm(c["a_codes"][None], c["a_scales"][None], c["a_alpha"],
                       c["b_codes"][None], c["b_scales"][None], c["b_alpha"])
        assert int(got[0, 0]) == c["bf16"], name


# K % 128 == 0 and K % 64 == 32 run the lane-dequantizing kernel (the latter
# with a partial last stage), K % 32 == 16 the workgroup-shared one, and
# K % 128 == 64 the lane kernel where its 128 x 128 tiles or its split last
# round apply (every small shape here, and the fourth split shape) and the
# shared one otherwise (4096 x 4096 x 320: one whole round of 256 x 256
# tiles); each list covers every case.  The lane kernel takes
# 128 x 128 tiles when there are too few 256 x 256 tiles to fill the chip
# (every small shape here) and 256 x 256 tiles otherwise (5376 x 5376: 441
# of them).  With 256 x 256 tiles, a last round of at most half the CUs'
# worth of tiles is split into K halves when K is long enough (SPLIT_SHAPES:
# 336 and 342 tiles, 80 and 86 left over, the second with a partial last
# stage and N % 8 != 0, the third with a half last stage).  A last round of
# at most a quarter of the CUs' worth runs as 128 x 128 quadrants of those
# tiles in a launch of their own (QUAD_SHAPES: 272, 289, 306 and 272 tiles,
# 16 to 50 left over, 12 or 13 K stages; the second with a partial last
# stage, the third ragged with N % 8 != 0, so that some quadrants fall
# outside the output, the fourth with a half last stage), and with at most
# an eighth and at least 16 K stages each quadrant as two K halves
# (QUAD_SPLIT_SHAPES: 16 left over; the second with a partial last stage,
# the third ragged with N % 8 != 0 and empty quadrants; 32 left over with a
# half last stage).
SPLIT_SHAPES = [(4096, 5376, 1536), (4353, 4700, 1440), (4096, 5376, 1600)]
QUAD_SHAPES = [(4352, 4096, 1536), (4352, 4200, 1440), (4353, 4100, 1536), (4352, 4096, 1600)]
QUAD_SPLIT_SHAPES = [(4352, 4096, 2048), (4352, 4096, 2080), (4224, 4001, 3072), (8192, 2240, 2240)]
# 128 x 128 tiles split too when K is long: 72 tiles of 24 and of 36
# stages, 72 of 18 (a half last stage), and a ragged 3 x 29 tiles with
# N % 8 != 0 (shapes whose 64 x 64 tiles fit in one round take the small kernel)
SMALL_SPLIT_SHAPES = [(384, 3072, 3072), (256, 4608, 4608), (512, 2240, 2240), (300, 3604, 4096)]


@pytest.mark.parametrize("M,N,K", [(1, 1, 16), (3, 5, 32), (37, 70, 64), (300, 260, 48),
                                   (257, 513, 16), (64, 96, 128), (300, 260, 256),
                                   (513, 700, 384), (64, 1000, 1280), (300, 260, 160),
                                   (513, 700, 224), (260, 300, 2240), (5376, 5376, 256),
                                   (5376, 5400, 96), (4200, 4360, 1120), (4096, 4096, 320)]
                        + SPLIT_SHAPES + QUAD_SHAPES + QUAD_SPLIT_SHAPES[:3] + SMALL_SPLIT_SHAPES)
def test_exact_sums_are_bit_exact(M, N, K):
    """Scales 1.0 and power-of-two alphas: every partial sum is a multiple of
    1/4 of magnitude at most 36 K < 2^16, exact in FP32 in any order, so the
    only rounding is the final BF16."""
    g = np.random.Generator(np.random.PCG64(M * 1000 + N + K))
    ac = g.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
    bc = g.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    as_ = np.full((M, K // 16), 0x38, np.uint8)
    bs = np.full((N, K // 16), 0x38, np.uint8)
    aa, ba = np.float32(2.0 ** -3), np.float32(2.0 ** 5)
    ref = O.nvfp4_gemm_ref(ac, as_, aa, bc, bs, ba)
    got = gpu_gemm(ac, as_, aa, bc, bs, ba)
    assert np.array_equal(got, O.bf16_output(ref))


@pytest.mark.parametrize("K", [224, 272, 384])
def test_one_hot_weight_returns_activation_columns(K):
    """B row n = code 0x2 (value 1) at k = n: the FP32 sum is the single
    product (s q)_A[m, n], exact, so out[m, n] = bf16(fp32(aA * (s q)_A[m, n]))
    bit for bit (the epilogue rounds alpha * acc + bias to FP32, then to
    BF16); pins nibble order, the [N, K] layout of B, scales and tails."""
    M, N = 300, 200
    ac, as_, aa = quantized("normal", M, K, 3)
    b4 = np.zeros((N, K), np.uint8)
    b4[np.arange(N), np.arange(N)] = 0x2
    bc = O.pack_codes(b4)
    bs = np.full((N, K // 16), 0x38, np.uint8)
    ref = O.nvfp4_gemm_ref(ac, as_, aa, bc, bs, np.float32(1.0))
    got = gpu_gemm(ac, as_, aa, bc, bs, np.float32(1.0))
    # ref is exact in float64 (24 + 6 significant bits); round as the epilogue
    # does: to FP32, then to BF16.  (alpha = amax/2688 has a periodic binary
    # mantissa, so FP32 results on a BF16 midpoint are common here and a
    # single rounding of ref would differ in a few percent of the outputs.)
    want = O.f64_to_bf16_bits_rne(ref.astype(np.float32).astype(np.float64))
    assert np.array_equal(got, want)


@pytest.mark.parametrize("K", [224, 272, 384])
@pytest.mark.parametrize("side", ["A", "B"])
def test_every_scale_code_bit_exact(side, K):
    """One operand cycles its block scales through all 127 finite E4M3 codes
    (subnormals included) with random codes; the other is one-hot (value 1 at
    k = row, scale 1.0).  Each output is a single exact product, so it must
    equal bf16(fp32(alpha * s * q)) bit for bit, on either operand side."""
    R = 300
    g = np.random.Generator(np.random.PCG64(31 if side == "A" else 32))
    c = g.integers(0, 256, size=(R, K // 2), dtype=np.uint8)
    sc = (np.arange(R * (K // 16)).reshape(R, K // 16) % 0x7F).astype(np.uint8)
    alpha = np.float32(0.37)
    n1 = 200
    h4 = np.zeros((n1, K), np.uint8)
    h4[np.arange(n1), np.arange(n1)] = 0x2
    hc = O.pack_codes(h4)
    hs = np.full((n1, K // 16), 0x38, np.uint8)
    if side == "A":
        args = (c, sc, alpha, hc, hs, np.float32(1.0))
    else:
        args = (hc, hs, np.float32(1.0), c, sc, alpha)
    ref = O.nvfp4_gemm_ref(*args)
    got = gpu_gemm(*args)
    want = O.f64_to_bf16_bits_rne(ref.astype(np.float32).astype(np.float64))
    assert np.array_equal(got, want)


@pytest.mark.parametrize("kind", ["wide", "blockscale"])
def test_wide_dynamic_range_vs_oracle(kind):
    """Operands whose blocks span many binades (tiny and subnormal E4M3
    scales, zero-scale blocks)."""
    g = np.random.Generator(np.random.PCG64(41))
    M, N, K = 300, 260, 1024
    from workloads import f32_to_bf16_bits

    def draw(rows):
        x = g.standard_normal((rows, K)).astype(np.float32)
        if kind == "wide":
            x *= np.exp2(g.integers(-24, 8, size=(rows, K))).astype(np.float32)
        else:
            x *= np.repeat(np.exp2(g.integers(-24, 7, size=(rows, K // 16))), 16, axis=1).astype(np.float32)
        return O.nvfp4_quantize_ref(f32_to_bf16_bits(x))
    a, b = draw(M), draw(N)
    assert (a[1] < 8).any() and (b[1] < 8).any()    # subnormal scales present
    ref = O.nvfp4_gemm_ref(*a, *b)
    got = gpu_gemm(*a, *b)
    err = rel_fro(got, ref)
    say(f"{kind}: rel_fro={err:.3e}")
    assert err <= TOL
    check_elements(got, a, b, ref)


# (64, 64, 128), (128, 1152, 1152), (96, 300, 3072), (1, 9, 128),
# (65, 130, 1152) and (200, 3000, 256) take the 64 x 64 kernel
SHAPES = [(1, 1, 16), (5, 7, 32), (64, 64, 128), (255, 257, 48), (300, 520, 272),
          (257, 129, 2240), (128, 1152, 1152), (513, 260, 5600), (96, 300, 3072),
          (260, 2049, 256), (513, 777, 640), (1, 9, 128), (65, 130, 1152), (200, 3000, 256),
          (2100, 9000, 3072)]   # 256 x 256 tiles


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("with_bias", [False, True])
def test_random_vs_oracle(M, N, K, with_bias):
    ac, as_, aa = quantized("normal", M, K, 7 * M + K)
    bc, bs, ba = quantized(None, N, K, 11 * N + K, sigma=0.02)
    bias = draw_bias(N, 0.02, N) if with_bias else None
    ref = O.nvfp4_gemm_ref(ac, as_, aa, bc, bs, ba, bias)
    got = gpu_gemm(ac, as_, aa, bc, bs, ba, bias)
    err = rel_fro(got, ref)
    mism = bf16_mismatch_fraction(got, ref)
    floor = rel_fro(O.bf16_output(ref), ref)
    say(f"M={M} N={N} K={K} bias={with_bias}: rel_fro={err:.3e} (bf16 floor {floor:.3e}) "
        f"mismatch={mism:.2e}")
    assert np.isfinite(O.bf16_bits_to_f32(got)).all()
    assert err <= TOL
    assert mism <= 0.01
    check_elements(got, (ac, as_, aa), (bc, bs, ba), ref, bias)


def test_zero_k_writes_bias():
    M, N = 33, 70
    bias = draw_bias(N, 0.5, 1)
    out = poison_bf16((M, N))
    z = torch.empty((M, 0), dtype=torch.uint8, device=device())
    zb = torch.empty((N, 0), dtype=torch.uint8, device=device())
    sol.nvfp4_gemm(z, z, f32_to_dev(1.0), zb, zb, f32_to_dev(1.0), bf16_to_dev(bias), out)
    torch.cuda.synchronize()
    assert np.array_equal(bf16_from_dev(out), np.broadcast_to(bias, (M, N)))


def test_route_lists_take_their_plans():
    for M, N, K in SPLIT_SHAPES:
        tiles = ((M + 255) // 256) * ((N + 255) // 256)
        assert sol.gemm_plan(M, N, K) == {"kernel": "nvfp4_gemm_lane_kernel", "tile": 256,
                                          "workgroups": tiles + tiles % 256, "splits": 2}
    for M, N, K in QUAD_SHAPES + QUAD_SPLIT_SHAPES:
        tiles = ((M + 255) // 256) * ((N + 255) // 256)
        splits = 2 if (M, N, K) in QUAD_SPLIT_SHAPES else 1
        rem = tiles % 256
        assert sol.gemm_plan(M, N, K) == {"kernel": "nvfp4_gemm_lane_kernel", "tile": 256,
                                          "workgroups": tiles - rem + 4 * rem * splits,
                                          "splits": splits}
        assert (sol.nvfp4_gemm_workspace_bytes(M, N, K) > 0) == (splits == 2)


@pytest.mark.parametrize("M,N,K", QUAD_SHAPES)
def test_quadrant_tail_vs_oracle(M, N, K):
    """The last round's tiles as whole 128 x 128 quadrants: the same bits as
    the same GEMM without a workspace (which takes the same plan) and as
    128 x 128 tiles would give (the same MFMAs per output element in the
    same order); within the bar of the oracle."""
    ac, as_, aa = quantized("normal", M, K, 7 * M + K)
    bc, bs, ba = quantized(None, N, K, 11 * N + K, sigma=0.02)
    bias = draw_bias(N, 0.02, N + 5)
    got = gpu_gemm(ac, as_, aa, bc, bs, ba, bias)
    assert np.array_equal(got, gpu_gemm(ac, as_, aa, bc, bs, ba, bias, split=False))
    ref = O.nvfp4_gemm_ref(ac, as_, aa, bc, bs, ba, bias)
    err = rel_fro(got, ref)
    say(f"quadrants M={M} N={N} K={K}: rel_fro={err:.3e}")
    assert err <= TOL
    assert bf16_mismatch_fraction(got, ref) <= 0.01
    check_elements(got, (ac, as_, aa), (bc, bs, ba), ref, bias, "quadrants ")


@pytest.mark.parametrize("M,N,K", SPLIT_SHAPES + QUAD_SPLIT_SHAPES + SMALL_SPLIT_SHAPES)
def test_split_last_round_vs_oracle(M, N, K):
    """The last round's tiles (or their quadrants) as two K halves: within
    the bar of the oracle, and the same bits on a second call (the workspace
    is reused, its counters cleared by the call itself) as on the first."""
    need = sol.nvfp4_gemm_workspace_bytes(M, N, K)
    assert need > 0
    ac, as_, aa = quantized("normal", M, K, 5 * M + K)
    bc, bs, ba = quantized(None, N, K, 3 * N + K, sigma=0.02)
    bias = draw_bias(N, 0.02, N)
    dev = device()
    args = [u8_to_dev(ac), u8_to_dev(as_), f32_to_dev(aa), u8_to_dev(bc), u8_to_dev(bs),
            f32_to_dev(ba), bf16_to_dev(bias)]
    ws = torch.full((need,), 0xA5, dtype=torch.uint8, device=dev)
    outs = []
    for _ in range(2):
        out = poison_bf16((M, N))
        sol.nvfp4_gemm(*args, out, workspace=ws)
        torch.cuda.synchronize()
        outs.append(bf16_from_dev(out))
    whole = gpu_gemm(ac, as_, aa, bc, bs, ba, bias, split=False)
    ref = O.nvfp4_gemm_ref(ac, as_, aa, bc, bs, ba, bias)
    err, err_whole = rel_fro(outs[0], ref), rel_fro(whole, ref)
    diff = float(np.mean(outs[0] != whole))
    say(f"split M={M} N={N} K={K}: rel_fro={err:.3e} (unsplit {err_whole:.3e}), "
        f"outputs differing from unsplit {diff:.2e}")
    assert np.array_equal(outs[0], outs[1])
    assert err <= TOL and err_whole <= TOL
    assert bf16_mismatch_fraction(outs[0], ref) <= 0.01
    check_elements(outs[0], (ac, as_, aa), (bc, bs, ba), ref, bias, "split ")
    check_elements(whole, (ac, as_, aa), (bc, bs, ba), ref, bias, "unsplit ")


@pytest.mark.parametrize("M,N,K", [SPLIT_SHAPES[0], QUAD_SPLIT_SHAPES[0], QUAD_SHAPES[0],
                                   SMALL_SPLIT_SHAPES[0]])
def test_split_gemm_in_a_replayed_graph(M, N, K):
    """A split GEMM captured once and replayed: the tile slots left by each
    replay (and by the eager calls between replays) must not confuse the
    next; every replay equals the eager result bit for bit."""
    ac, as_, aa = quantized("normal", M, K, 17)
    bc, bs, ba = quantized(None, N, K, 19, sigma=0.02)
    args = [u8_to_dev(ac), u8_to_dev(as_), f32_to_dev(aa), u8_to_dev(bc), u8_to_dev(bs),
            f32_to_dev(ba), None]
    dev = device()
    ws = torch.empty(sol.nvfp4_gemm_workspace_bytes(M, N, K), dtype=torch.uint8, device=dev)
    eager = poison_bf16((M, N))
    sol.nvfp4_gemm(*args, eager, workspace=ws)
    torch.cuda.synchronize()
    want = bf16_from_dev(eager)
    out = poison_bf16((M, N))
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):   # warm-up on the capture stream, as torch asks
        sol.nvfp4_gemm(*args, out, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sol.nvfp4_gemm(*args, out, workspace=ws)
    for _ in range(3):
        out.view(torch.int16).fill_(0x7FC1)
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bf16_from_dev(out), want)
        sol.nvfp4_gemm(*args, eager, workspace=ws)
        torch.cuda.synchronize()
        assert np.array_equal(bf16_from_dev(eager), want)


def test_deterministic():
    M, N, K = 1000, 1500, 3072
    ac, as_, aa = quantized("normal", M, K, 1)
    bc, bs, ba = quantized(None, N, K, 2, sigma=0.015)
    r1 = gpu_gemm(ac, as_, aa, bc, bs, ba)
    r2 = gpu_gemm(ac, as_, aa, bc, bs, ba)
    assert np.array_equal(r1, r2)


@pytest.mark.parametrize("M,N,K", [(256, 3072, 1152), (200, 2050, 640), (200, 3000, 256)])
def test_small_tiles_match_the_lane_kernel(M, N, K):
    """The 64 x 64 kernel uses the lane kernel's dequantization, K order and
    epilogue, so it must give the lane kernel's output bit for bit.  The
    lane kernel is reached with the same operands padded by 64 zero
    elements along K (codes 0 under scale 0): K % 128 == 64 does not take
    the small kernel, and the padding adds only exact zeros to every sum."""
    import paper_2604_06916_amd as sol2
    assert sol2.gemm_plan(M, N, K)["kernel"] == "nvfp4_gemm_small_kernel"
    assert sol2.gemm_plan(M, N, K + 64, with_workspace=False)["kernel"] == "nvfp4_gemm_lane_kernel"
    ac, as_, aa = quantized("normal", M, K, 13)
    bc, bs, ba = quantized(None, N, K, 14, sigma=0.02)
    small = gpu_gemm(ac, as_, aa, bc, bs, ba)

    def pad(c, sc):
        return np.pad(c, ((0, 0), (0, 32))), np.pad(sc, ((0, 0), (0, 4)))
    (acp, asp), (bcp, bsp) = pad(ac, as_), pad(bc, bs)
    lane = gpu_gemm(acp, asp, aa, bcp, bsp, ba, split=False)
    assert np.array_equal(small, lane)
    ref = O.nvfp4_gemm_ref(ac, as_, aa, bc, bs, ba)
    assert rel_fro(small, ref) <= TOL
    check_elements(small, (ac, as_, aa), (bc, bs, ba), ref)


# Few tokens on the wave-K kernel (32 x 32 tiles, the K stages of a
# workgroup dealt to its four waves, their sums added in LDS in wave
# order): 1 stage (three waves without one), 3, 5 (uneven shares), 9 and 36
# stages; ragged M and N, N % 8 != 0; 384 tiles, so that two workgroups
# share a CU.  The exact-sum shapes (64, 96, 128), (300, 260, 256) and
# (64, 1000, 1280) above take this kernel too.
WAVEK_SHAPES = [(7, 33, 128), (100, 200, 384), (33, 40, 640), (65, 130, 1152),
                (128, 1152, 1152), (128, 1152, 4608), (128, 3072, 3072)]


@pytest.mark.parametrize("M,N,K", WAVEK_SHAPES)
def test_wavek_kernel_vs_oracle(M, N, K):
    assert sol.gemm_plan(M, N, K)["kernel"] == "nvfp4_gemm_wavek_kernel"
    ac, as_, aa = quantized("outlier4x20", M, K, 21 * M + K)
    bc, bs, ba = quantized(None, N, K, 23 * N + K, sigma=0.02)
    bias = draw_bias(N, 0.02, N + 1)
    got = gpu_gemm(ac, as_, aa, bc, bs, ba, bias)
    assert np.array_equal(got, gpu_gemm(ac, as_, aa, bc, bs, ba, bias))   # fixed sum order
    ref = O.nvfp4_gemm_ref(ac, as_, aa, bc, bs, ba, bias)
    err = rel_fro(got, ref)
    say(f"M={M} N={N} K={K}: rel_fro={err:.3e}")
    assert err <= TOL
    check_elements(got, (ac, as_, aa), (bc, bs, ba), ref, bias)


@pytest.mark.parametrize("M,N,K", [(7, 33, 128), (33, 40, 640), (128, 1152, 4608)])
def test_wavek_exact_sums_are_bit_exact(M, N, K):
    """As test_exact_sums_are_bit_exact, on the wave-K kernel."""
    assert sol.gemm_plan(M, N, K)["kernel"] == "nvfp4_gemm_wavek_kernel"
    g = np.random.Generator(np.random.PCG64(M * 1000 + N + K))
    ac = g.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
    bc = g.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    as_ = np.full((M, K // 16), 0x38, np.uint8)
    bs = np.full((N, K // 16), 0x38, np.uint8)
    aa, ba = np.float32(2.0 ** -3), np.float32(2.0 ** 5)
    ref = O.nvfp4_gemm_ref(ac, as_, aa, bc, bs, ba)
    got = gpu_gemm(ac, as_, aa, bc, bs, ba)
    assert np.array_equal(got, O.bf16_output(ref))
