"""Pins for the CPU oracle (no GPU).

The oracle is checked against things other than itself: the format
definitions enumerated exhaustively, hand-worked tensors (tests/golden), an
exact-rational scalar re-implementation (exact_ref.py), closed forms and
invariants.  The last group plants plausible mistakes in the oracle and checks
that at least one pin catches each.
"""
import math

import numpy as np
import pytest

import exact_ref as X
import golden_io
import oracle.nvfp4 as O

F = X.F


def bf16(vals):
    return golden_io.f32_to_bf16_exact(np.asarray(vals, dtype=np.float32))


# ---------------------------------------------------------------------------
# Pins written as plain functions so the mutation tests can re-run them
# against a deliberately broken oracle.
# ---------------------------------------------------------------------------

def pin_e2m1_table():
    # Preliminaries: 1 sign, 2 exponent (bias 1), 1 mantissa bit.
    expect = [0, .5, 1, 1.5, 2, 3, 4, 6, -0.0, -.5, -1, -1.5, -2, -3, -4, -6]
    got = O.e2m1_decode(np.arange(16))
    assert np.array_equal(got, np.array(expect))
    assert np.array_equal(np.signbit(got), np.arange(16) >= 8)
    assert [float(v) for v in X.E2M1] == expect[:8]


def pin_e2m1_midpoints():
    # (value, expected magnitude code): ties go to the even code.
    cases = [(0.25, 0), (0.75, 2), (1.25, 2), (1.75, 4), (2.5, 4), (3.5, 6), (5.0, 6),
             (6.0, 7), (6.375, 7), (1e30, 7), (0.0, 0), (0.5, 1), (3.0, 5)]
    for v, c in cases:
        v32 = np.float32(v)
        assert O.e2m1_encode_rne_sat(v32) == c, (v, c)
        assert O.e2m1_encode_rne_sat(-v32) == c | 8, (-v, c)
        if 0 < v < 6:
            below = np.nextafter(v32, np.float32(0))
            above = np.nextafter(v32, np.float32(100))
            lo_code = X.nearest_code(F(float(below)), X.E2M1)
            hi_code = X.nearest_code(F(float(above)), X.E2M1)
            assert O.e2m1_encode_rne_sat(below) == lo_code
            assert O.e2m1_encode_rne_sat(above) == hi_code
    # the six midpoints that are not ties-to-even of 0.25 are distinct cases
    assert O.e2m1_encode_rne_sat(np.nextafter(np.float32(0.25), np.float32(1))) == 1
    assert O.e2m1_encode_rne_sat(np.nextafter(np.float32(0.75), np.float32(0))) == 1


def pin_e4m3_table():
    vals = O.e4m3_decode(np.arange(256))
    nan = np.isnan(vals)
    assert list(np.nonzero(nan)[0]) == [0x7F, 0xFF]
    anchors = {0x00: 0.0, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x08: 2.0 ** -6,
               0x38: 1.0, 0x50: 8.0, 0x51: 9.0, 0x52: 10.0, 0x78: 256.0, 0x7E: 448.0}
    for c, v in anchors.items():
        assert vals[c] == v, hex(c)
        assert vals[c | 0x80] == -v or (v == 0 and np.signbit(vals[0x80]))
    pos = vals[:0x7F]
    assert np.all(np.diff(pos) > 0)
    assert [F(float(v)) for v in pos] == X.E4M3


def pin_e4m3_encode():
    table = O.e4m3_decode(np.arange(0x7F))
    # every non-negative finite value round-trips
    assert np.array_equal(O.e4m3_encode_rne_sat(table.astype(np.float32)), np.arange(0x7F))
    # every midpoint goes to the even code; its neighbours go to the nearer one
    for c in range(0x7E):
        mid = np.float32((table[c] + table[c + 1]) / 2)
        assert float(mid) == (table[c] + table[c + 1]) / 2  # exact in binary32
        even = c if c % 2 == 0 else c + 1
        assert O.e4m3_encode_rne_sat(mid) == even, hex(c)
        assert O.e4m3_encode_rne_sat(np.nextafter(mid, np.float32(0))) == c
        assert O.e4m3_encode_rne_sat(np.nextafter(mid, np.float32(1e9))) == c + 1
    fixed = {2.0 ** -10: 0x00, 7.5 * 2.0 ** -9: 0x08, 8.5: 0x50, 9.5: 0x52, 448.0: 0x7E,
             464.0: 0x7E, 1e30: 0x7E, 0.0: 0x00}
    for v, c in fixed.items():
        assert O.e4m3_encode_rne_sat(np.float32(v)) == c, v
    assert O.e4m3_encode_rne_sat(np.nextafter(np.float32(2.0 ** -10), np.float32(1))) == 0x01


def pin_golden_quantize():
    cases = golden_io.load()
    for name, c in cases.items():
        if c["kind"] != "case":
            continue
        codes, scales, alpha = O.nvfp4_quantize_ref(bf16(c["x"])[None, :])
        assert codes.tobytes() == c["codes"].tobytes(), name
        assert scales.tobytes() == c["scales"].tobytes(), name
        assert np.float32(alpha).view(np.uint32) == np.float32(c["alpha"]).view(np.uint32), name


def pin_golden_gemm():
    cases = golden_io.load()
    for name, c in cases.items():
        if c["kind"] != "gemm":
            continue
        out = O.nvfp4_gemm_ref(c["a_codes"][None], c["a_scales"][None], c["a_alpha"],
                               c["b_codes"][None], c["b_scales"][None], c["b_alpha"])
        assert out[0, 0] == c["exact"], name
        assert int(O.bf16_output(out)[0, 0]) == c["bf16"], name


def _tiny_tensor(g, rows, K, kind):
    if kind == "normal":
        x = g.standard_normal((rows, K)).astype(np.float32)
    elif kind == "dyadic":        # few distinct values: exact ties are frequent
        x = (g.integers(-24, 25, size=(rows, K)) * 0.125).astype(np.float32)
    elif kind == "wide":          # blocks spanning many binades, some underflowing
        x = (g.standard_normal((rows, K)) * np.exp2(g.integers(-30, 8, size=(rows, K)))).astype(np.float32)
    elif kind == "blockscale":    # per-block magnitudes 2^-20 .. 2^6
        x = g.standard_normal((rows, K)).astype(np.float32)
        x *= np.repeat(np.exp2(g.integers(-20, 7, size=(rows, K // 16))), 16, axis=1).astype(np.float32)
    elif kind == "midpoint":
        # alpha = 5.25/2688 = 2^-9 is fixed by one element; every other block
        # has amax 6 d with d = s 2^-9 for a random normal E4M3 s, so its scale
        # is exactly s, and its elements are E2M1 midpoints times d: exact ties
        # of x/d that x * RN(1/d) may or may not keep.
        mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
        x = np.zeros((rows, K), np.float32)
        for r_ in range(rows):
            for b in range(K // 16):
                s = float(O.e4m3_decode(int(g.integers(0x08, 0x7F))))
                d = s * 2.0 ** -9
                blk = np.concatenate([[6.0], mids, g.choice(mids, 8)]) * d
                blk *= np.where(g.random(16) < 0.5, -1.0, 1.0)
                x[r_, 16 * b:16 * b + 16] = blk
        x[0, 0] = 5.25
    else:
        raise ValueError(kind)
    from workloads import f32_to_bf16_bits
    return f32_to_bf16_bits(x)


def pin_exact_reference(n_cases=30, seed=7):
    g = np.random.Generator(np.random.PCG64(seed))
    kinds = ["normal", "dyadic", "wide", "blockscale", "midpoint"]
    for i in range(n_cases):
        rows = int(g.integers(1, 4))
        K = 16 * int(g.integers(1, 5))
        xb = _tiny_tensor(g, rows, K, kinds[i % len(kinds)])
        codes, scales, alpha = O.nvfp4_quantize_ref(xb)
        ecodes, escales, ealpha = X.quantize_exact([[int(v) for v in r] for r in xb])
        assert F(float(alpha)) == ealpha, i
        assert np.array_equal(scales, np.array(escales, dtype=np.uint8)), i
        assert np.array_equal(O.unpack_codes(codes), np.array(ecodes, dtype=np.uint8)), i


def pin_gemm_exact(seed=11):
    g = np.random.Generator(np.random.PCG64(seed))
    for i in range(12):
        M, N = int(g.integers(1, 6)), int(g.integers(1, 6))
        K = 16 * int(g.integers(1, 4))
        ac = g.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
        bc = g.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
        as_ = g.integers(0, 0x7F, size=(M, K // 16), dtype=np.uint8)
        bs = g.integers(0, 0x7F, size=(N, K // 16), dtype=np.uint8)
        aa = np.float32(g.uniform(0.01, 2))
        ba = np.float32(g.uniform(0.01, 2))
        bias = bf16(np.round(g.standard_normal(N) * 64) / 64) if i % 2 else None
        out = O.nvfp4_gemm_ref(ac, as_, aa, bc, bs, ba, bias)
        ex = X.gemm_exact(O.unpack_codes(ac).tolist(), as_.tolist(), F(float(aa)),
                          O.unpack_codes(bc).tolist(), bs.tolist(), F(float(ba)),
                          None if bias is None else [F(float(v)) for v in O.bf16_bits_to_f32(bias)])
        for m in range(M):
            for n in range(N):
                e = float(ex[m][n])
                assert abs(out[m, n] - e) <= 1e-14 * max(1.0, abs(e)), (i, m, n)


def pin_gemm_one_hot(seed=5):
    # B row n holds code 0x2 (value 1) at k = n and 0 elsewhere, scales 1.0,
    # alpha_B = 1: the product returns the decoded columns 0..N-1 of A.  Pins
    # the nibble order, the [N, K] layout of B and the block-to-scale mapping.
    g = np.random.Generator(np.random.PCG64(seed))
    M, N, K = 5, 40, 48
    xb = _tiny_tensor(g, M, K, "normal")
    ac, as_, aa = O.nvfp4_quantize_ref(xb)
    b4 = np.zeros((N, K), dtype=np.uint8)
    b4[np.arange(N), np.arange(N)] = 0x2
    bc = O.pack_codes(b4)
    bs = np.full((N, K // 16), 0x38, dtype=np.uint8)
    out = O.nvfp4_gemm_ref(ac, as_, aa, bc, bs, np.float32(1.0))
    deq = O.nvfp4_dequantize_ref(ac, as_, aa)
    assert np.array_equal(out, deq[:, :N])
    # and decoding agrees element by element with the exact scalar decode
    u = O.unpack_codes(ac)
    for m in range(M):
        for k in range(K):
            assert F(float(deq[m, k])) == F(float(aa)) * X.decode_exact(int(u[m, k]), int(as_[m, k // 16]))


def pin_invariants(seed=3):
    g = np.random.Generator(np.random.PCG64(seed))
    xb = _tiny_tensor(g, 4, 64, "normal")
    c0, s0, a0 = O.nvfp4_quantize_ref(xb)
    x = O.bf16_bits_to_f32(xb)
    from workloads import f32_to_bf16_bits
    # (i) power-of-two scaling leaves codes and scales alone, scales alpha
    for k in (-7, -1, 3, 9):
        ck, sk, ak = O.nvfp4_quantize_ref(f32_to_bf16_bits(x * np.float32(2.0 ** k)))
        assert np.array_equal(ck, c0) and np.array_equal(sk, s0)
        assert ak == np.float32(a0 * np.float32(2.0 ** k))
    # (ii) sign symmetry: negation flips only the sign bits
    cn, sn, an = O.nvfp4_quantize_ref(xb ^ np.uint16(0x8000))
    assert an == a0 and np.array_equal(sn, s0)
    assert np.array_equal(cn, c0 ^ np.uint8(0x88))
    # (iii) block locality: editing one block below amax changes only it
    xe = x.copy()
    xe[2, 16:32] = x[2, 16:32] * np.float32(0.25)
    ce, se, ae = O.nvfp4_quantize_ref(f32_to_bf16_bits(xe))
    assert ae == a0
    mask_b = np.ones_like(s0, bool)
    mask_b[2, 1] = False
    assert np.array_equal(se[mask_b], s0[mask_b])
    mask_c = np.ones_like(c0, bool)
    mask_c[2, 8:16] = False
    assert np.array_equal(ce[mask_c], c0[mask_c])
    # (iv) error bound: |x - alpha s q| <= alpha s h(|y|) + saturation excess
    deq = O.nvfp4_dequantize_ref(c0, s0, a0)
    s = np.repeat(O.e4m3_decode(s0), 16, axis=1)
    unit = np.float64(a0) * s
    with np.errstate(divide="ignore", invalid="ignore"):
        y = np.abs(x) / unit
    assert np.all(unit > 0)
    h = np.where(y < 2, 0.25, np.where(y < 4, 0.5, 1.0)) + np.maximum(y - 6, 0)
    assert np.all(np.abs(x - deq) <= unit * h * (1 + 1e-6))


def pin_bf16_rounding(seed=13):
    g = np.random.Generator(np.random.PCG64(seed))
    v = g.standard_normal(300) * np.exp2(g.integers(-140, 120, size=300))
    ties = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(2 + 2.0 ** -7), 2.0 ** -134, 3 * 2.0 ** -134])
    v = np.concatenate([v, ties])
    got = O.f64_to_bf16_bits_rne(v)
    for val, bits in zip(v, got):
        # exact: binary32 rounding with a 8-bit significand, from the definition
        a = abs(F(float(val)))
        e = max(X._floor_log2(a), -126) if a else -126
        q = F(2) ** (e - 7)
        r = X._round_half_even(a / q) * q
        want = float(r) if val >= 0 else -float(r)
        have = float(O.bf16_bits_to_f32(np.array([bits], np.uint16))[0])
        assert have == want or (math.isinf(have) and r >= 2 ** 128), val


def pin_e8m0_table():
    v = O.e8m0_decode(np.arange(256))
    assert np.isnan(v[255]) and not np.isnan(v[:255]).any()
    assert v[127] == 1.0 and v[0] == 2.0 ** -127 and v[254] == 2.0 ** 127 and v[124] == 0.125
    assert np.all(np.diff(v[:255]) > 0)


def pin_golden_mx():
    cases = golden_io.load()
    for name, c in cases.items():
        if c["kind"] == "mxcase":
            codes, scales = O.mxfp4_quantize_ref(bf16(c["x"])[None, :])
            assert codes.tobytes() == c["codes"].tobytes(), name
            assert scales.tobytes() == c["mxscales"].tobytes(), name
        elif c["kind"] == "mxgemm":
            out = O.mxfp4_gemm_ref(c["a_codes"][None], c["a_scales"][None],
                                   c["b_codes"][None], c["b_scales"][None])
            assert out[0, 0] == c["exact"], name
            assert int(O.bf16_output(out)[0, 0]) == c["bf16"], name


def pin_mx_exact_reference(seed=19):
    g = np.random.Generator(np.random.PCG64(seed))
    kinds = ["normal", "dyadic", "wide", "blockscale"]
    for i in range(16):
        rows = int(g.integers(1, 4))
        K = 32 * int(g.integers(1, 3))
        xb = _tiny_tensor(g, rows, K, kinds[i % len(kinds)])
        codes, scales = O.mxfp4_quantize_ref(xb)
        ec, es = X.mx_quantize_exact([[int(v) for v in r] for r in xb])
        assert np.array_equal(scales, np.array(es, dtype=np.uint8)), i
        assert np.array_equal(O.unpack_codes(codes), np.array(ec, dtype=np.uint8)), i


def pin_mx_gemm_exact(seed=23):
    g = np.random.Generator(np.random.PCG64(seed))
    for i in range(8):
        M, N = int(g.integers(1, 5)), int(g.integers(1, 5))
        K = 32 * int(g.integers(1, 3))
        ac = g.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
        bc = g.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
        as_ = g.integers(100, 150, size=(M, K // 32), dtype=np.uint8)
        bs = g.integers(100, 150, size=(N, K // 32), dtype=np.uint8)
        bias = bf16(np.round(g.standard_normal(N) * 64) / 64) if i % 2 else None
        out = O.mxfp4_gemm_ref(ac, as_, bc, bs, bias)
        ex = X.mx_gemm_exact(O.unpack_codes(ac).tolist(), as_.tolist(), O.unpack_codes(bc).tolist(),
                             bs.tolist(), None if bias is None else [F(float(v)) for v in O.bf16_bits_to_f32(bias)])
        for m in range(M):
            for n in range(N):
                e = float(ex[m][n])
                assert abs(out[m, n] - e) <= 1e-14 * max(1.0, abs(e)), (i, m, n)


def pin_mx_invariants(seed=29):
    g = np.random.Generator(np.random.PCG64(seed))
    xb = _tiny_tensor(g, 3, 64, "normal")
    c0, s0 = O.mxfp4_quantize_ref(xb)
    x = O.bf16_bits_to_f32(xb)
    from workloads import f32_to_bf16_bits
    for k in (-5, 3, 11):
        ck, sk = O.mxfp4_quantize_ref(f32_to_bf16_bits(x * np.float32(2.0 ** k)))
        assert np.array_equal(ck, c0) and np.array_equal(sk.astype(int), s0.astype(int) + k)
    cn, sn = O.mxfp4_quantize_ref(xb ^ np.uint16(0x8000))
    assert np.array_equal(sn, s0) and np.array_equal(cn, c0 ^ np.uint8(0x88))
    # every block's largest magnitude decodes within [4, 8) * 2^E and
    # elements round to within half an E2M1 step of x / 2^E (or saturate)
    deq = O.mxfp4_unscaled_ref(c0, s0)
    X_ = np.repeat(O.e8m0_decode(s0), 32, axis=1)
    y = np.abs(x) / X_
    assert np.all((y.reshape(3, 2, 32).max(axis=2) >= 4) & (y.reshape(3, 2, 32).max(axis=2) < 8))
    h = np.where(y < 2, 0.25, np.where(y < 4, 0.5, 1.0)) + np.maximum(y - 6, 0)
    assert np.all(np.abs(x - deq) <= X_ * h * (1 + 1e-9))


ALL_PINS = [pin_e8m0_table, pin_golden_mx, pin_mx_exact_reference, pin_mx_gemm_exact,
            pin_mx_invariants, pin_e2m1_table, pin_e2m1_midpoints, pin_e4m3_table, pin_e4m3_encode,
            pin_golden_quantize, pin_golden_gemm, pin_exact_reference, pin_gemm_exact,
            pin_gemm_one_hot, pin_invariants, pin_bf16_rounding]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin()


def test_e2m1_encoder_all_small_bf16():
    """Every non-negative BF16 value below 8 through the E2M1 encoder vs the
    exact nearest-value search."""
    bits = np.arange(0, 0x4100, dtype=np.uint16)  # 0 .. 8.0
    y = O.bf16_bits_to_f32(bits)
    got = O.e2m1_encode_rne_sat(y)
    want = np.array([X.nearest_code(F(float(v)), X.E2M1) for v in y], dtype=np.uint8)
    assert np.array_equal(got, want)


def test_e4m3_encoder_log_sweep():
    g = np.random.Generator(np.random.PCG64(17))
    v = np.exp2(g.uniform(-12, 10, size=3000)).astype(np.float32)
    got = O.e4m3_encode_rne_sat(v)
    want = np.array([X.nearest_code(F(float(t)), X.E4M3) for t in v], dtype=np.uint8)
    assert np.array_equal(got, want)


def test_quantize_rejects_bad_shapes():
    with pytest.raises(ValueError):
        O.nvfp4_quantize_ref(np.zeros((2, 24), np.uint16))
    with pytest.raises(ValueError):
        O.nvfp4_quantize_ref(np.zeros(32, np.uint16))


def test_empty_tensor():
    c, s, a = O.nvfp4_quantize_ref(np.zeros((0, 32), np.uint16))
    assert c.shape == (0, 16) and s.shape == (0, 2) and a == 0


# ---------------------------------------------------------------------------
# Planted mistakes: each must make at least one pin fail.
# ---------------------------------------------------------------------------

def _any_pin_fails():
    for pin in ALL_PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            return True
    return False


def _mut_nibble_order(mp):
    mp.setattr(O, "pack_codes", lambda c: (np.asarray(c)[..., 1::2] & 0xF) | ((np.asarray(c)[..., 0::2] & 0xF) << 4))


def _mut_ties_away(mp):
    orig = O._round_to_table_rne

    def ties_up(v, table):
        v = np.asarray(v, dtype=np.float64)
        idx = orig(v, table)
        lo = np.clip(np.searchsorted(table, v, side="right") - 1, 0, len(table) - 1)
        hi = np.minimum(lo + 1, len(table) - 1)
        tie = v == (table[lo] + table[hi]) / 2
        return np.where(tie & (v < table[-1]), hi, idx)
    mp.setattr(O, "_round_to_table_rne", ties_up)


def _mut_alpha_divisor(mp):
    mp.setattr(O, "ALPHA_DIVISOR", np.float32(6.0 * 447.0))


def _mut_division_order(mp):
    # y = x / (s alpha) by division instead of multiply-by-reciprocal
    orig = O.nvfp4_quantize_ref

    def variant(x_bits):
        x_bits = np.asarray(x_bits, dtype=np.uint16)
        c, s, a = orig(x_bits)
        if a == 0:
            return c, s, a
        rows, K = x_bits.shape
        x = O.bf16_bits_to_f32(x_bits).reshape(rows, K // 16, 16)
        d = (O.e4m3_decode(s).astype(np.float32) * a).astype(np.float32)
        with np.errstate(divide="ignore", invalid="ignore"):
            y = (x / d[:, :, None]).astype(np.float32)
        q = O.e2m1_encode_rne_sat(y, sign_source=x)
        q = np.where((s == 0)[:, :, None], (np.signbit(x).astype(np.uint8) << 3), q)
        return O.pack_codes(q.reshape(rows, K)), s, a
    mp.setattr(O, "nvfp4_quantize_ref", variant)


def _mut_transposed_b(mp):
    # B read as if stored [K, N] instead of [N, K]
    orig = O.nvfp4_unscaled_ref

    def gemm(a_codes, a_scales, a_alpha, b_codes, b_scales, b_alpha, bias_bits=None):
        aq = orig(a_codes, a_scales)
        bq = orig(b_codes, b_scales)
        acc = aq @ bq.reshape(bq.shape[1], bq.shape[0])
        out = np.float64(a_alpha) * np.float64(b_alpha) * acc
        if bias_bits is not None:
            out = out + O.bf16_bits_to_f32(bias_bits).astype(np.float64)[None, :]
        return out
    mp.setattr(O, "nvfp4_gemm_ref", gemm)


def _mut_dropped_bias(mp):
    orig = O.nvfp4_gemm_ref
    mp.setattr(O, "nvfp4_gemm_ref", lambda *a, **k: orig(*a[:6]))


def _mut_scale_per_32(mp):
    orig = O.nvfp4_unscaled_ref

    def per32(codes, scales):
        s = np.asarray(scales).copy()
        s[:, 1::2] = s[:, 0::2][:, :s[:, 1::2].shape[1]]
        return orig(codes, s)
    mp.setattr(O, "nvfp4_unscaled_ref", per32)


def _mut_e4m3_bias(mp):
    orig = O.e4m3_decode
    mp.setattr(O, "e4m3_decode", lambda c: orig(c) * 2.0)


def _mut_mx_exponent_offset(mp):
    # shared exponent floor(log2 amax) - 1 instead of - 2

    def variant(x_bits):
        x_bits = np.asarray(x_bits, dtype=np.uint16)
        rows, K = x_bits.shape
        x = O.bf16_bits_to_f32(x_bits).astype(np.float64).reshape(rows, K // 32, 32)
        amax = np.abs(x).max(axis=2)
        _, e = np.frexp(np.where(amax > 0, amax, 1.0))
        code = np.where(amax > 0, np.clip(e - 1 - 1 + 127, 0, 254), 0)
        y = x / np.exp2(code - 127.0)[:, :, None]
        q = O.e2m1_encode_rne_sat(y.astype(np.float32), sign_source=x.astype(np.float32))
        return O.pack_codes(q.reshape(rows, K)), code.astype(np.uint8)
    mp.setattr(O, "mxfp4_quantize_ref", variant)


def _mut_mx_scale_broadcast(mp):
    # scale broadcast along the wrong axis: element k takes scale k mod (K/32)
    def variant(codes, scales):
        q = O.e2m1_decode(O.unpack_codes(codes))
        rows, K = q.shape
        return q * np.tile(O.e8m0_decode(scales), (1, 32))[:, :K]
    mp.setattr(O, "mxfp4_unscaled_ref", variant)


@pytest.mark.parametrize("mutation", [_mut_nibble_order, _mut_ties_away, _mut_alpha_divisor,
                                      _mut_division_order, _mut_transposed_b, _mut_dropped_bias,
                                      _mut_scale_per_32, _mut_e4m3_bias,
                                      _mut_mx_exponent_offset, _mut_mx_scale_broadcast],
                         ids=lambda f: f.__name__[5:])
def test_planted_mistake_is_caught(monkeypatch, mutation):
    assert not _any_pin_fails()
    mutation(monkeypatch)
    assert _any_pin_fails()
