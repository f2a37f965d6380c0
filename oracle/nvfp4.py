"""CPU oracle for the NVFP4 linear-layer hot path (Sol-RL, arXiv 2604.06916).

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow, obviously-correct
statement of what the GPU library computes.  Only the test suite, the smoke
check and the CPU-baseline leg of the benchmark may import it.  It shares no
code with the HIP library and never imports it; the library never imports it.

What is computed, and where the paper fixes it
----------------------------------------------
Preliminaries, "FP4 Quantization and Hardware Acceleration" (the paragraph
before the Methodology section) defines the method:

* an FP4 element has 1 sign, 2 exponent and 1 mantissa bit (E2M1);
* contiguous elements share one scale (block micro-scaling); NVIDIA's NVFP4
  groups 16 elements under an E4M3 scale, OCP MXFP4 groups 32 under E8M0;
* quantization is  x~ = Q(x) = S * Pi_FP4(x / S),  S the shared scale and
  Pi_FP4 the projection onto the FP4 grid.

Sec. 3.4 ("FP4-Empowered Two-Stage Framework", Stage 1) and Sec. 4.1 use this
quantizer for the weights and activations of every linear layer of the
denoiser, whose products run as "NVFP4 dense operations".

The paper is silent on the rest; this oracle takes the following readings
(all listed, with reasons, in the design notes):

R1  A second, per-tensor FP32 decode scale  alpha = amax(|x|) / (6 * 448),
    so a stored element decodes to  alpha * s * q  (s: E4M3 block scale,
    q: E2M1 value).
R2  One fixed IEEE-754 binary32 operation order (round to nearest even at
    every step), in this order:
      alpha = amax_g / 2688
      t     = alpha * 6
      s_f   = amax_b / t                       (amax_b: max |x| of the block)
      s     = E4M3_RNE_SAT(s_f)
      d     = s * alpha
      r     = 1 / d
      y     = x * r
      q     = E2M1_RNE_SAT(y)                  (sign of x kept, also on zero)
R3  E4M3 rounding: nearest value, ties to the even code, values at or above
    448 saturate to 448 (0x7E); E2M1 rounding likewise, saturating at 6.
R4  amax_g == 0 gives alpha = 0, all scales 0 and all codes = sign << 3; a
    block whose scale rounds to 0 gets codes = sign << 3.
R5  Layout: row-major; byte j of a code row holds element 2j in bits 3:0 and
    element 2j+1 in bits 7:4; scales row-major [rows][K/16].
R6  GEMM:  out[m, n] = bf16_rne( alpha_A * alpha_B * sum_k (s_A q_A)(s_B q_B)
    + bias[n] ), B stored [N, K] (nn.Linear layout).  The oracle evaluates the
    sum in float64 on exactly dequantized operands.

MXFP4 (the OCP variant named beside NVFP4 in the same paragraph: 32
elements under one E8M0 scale) follows the OCP MX conversion rule:
RM1 shared exponent E = floor(log2(amax_b)) - 2 (2 = largest E2M1
    exponent), scale 2^E stored as the E8M0 byte E + 127 clamped to
    [0, 254]; an all-zero block stores 0 (2^-127);
RM2 q = E2M1_RNE_SAT(x / 2^E), sign kept on zero (x / 2^E is exact);
RM3 no per-tensor scale; GEMM out = bf16_rne(sum_k (X_A q_A)(X_B q_B) + bias).

Every function below cites the passage or reading it follows.  Parity of the
quantizer is pinned by hand-worked tensors, exhaustive format tables, an
exact-rational scalar re-implementation and invariants (tests/); the GEMM by
closed forms and exact-rational brute force.
"""
from __future__ import annotations

import numpy as np

# ---------------------------------------------------------------------------
# Formats (Preliminaries: E2M1 element, E4M3 NVFP4 scale, E8M0 MXFP4 scale)
# ---------------------------------------------------------------------------

#: E2M1 magnitudes for codes 0..7 (1 sign, 2 exponent bits with bias 1,
#: 1 mantissa bit; exponent field 0 is subnormal: 0 and 0.5).
E2M1_MAGNITUDES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)

#: Largest finite E4M3 (OCP "E4M3FN": no infinities, 0x7F / 0xFF are NaN).
E4M3_MAX = 448.0
#: Per-tensor scale divisor of reading R1: largest E2M1 times largest E4M3.
ALPHA_DIVISOR = np.float32(6.0 * 448.0)
NVFP4_BLOCK = 16
MXFP4_BLOCK = 32


def e2m1_decode(codes) -> np.ndarray:
    """Value of 4-bit E2M1 codes (bit 3 = sign), float64.  Preliminaries."""
    c = np.asarray(codes, dtype=np.uint8)
    mag = E2M1_MAGNITUDES[c & 7]
    return np.where((c & 8) != 0, -mag, mag)


def e4m3_decode(codes) -> np.ndarray:
    """Value of E4M3 bytes, float64 (NaN for 0x7F/0xFF).  Preliminaries (NVFP4
    block scale); bit layout of the OCP FP8 E4M3 format: bias 7, exponent
    field 0 subnormal, no infinities."""
    b = np.asarray(codes, dtype=np.int64)
    sign = np.where((b >> 7) & 1, -1.0, 1.0)
    e = (b >> 3) & 0xF
    m = b & 7
    normal = (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7.0)
    sub = (m / 8.0) * 2.0 ** -6
    v = np.where(e == 0, sub, normal)
    v = np.where((e == 15) & (m == 7), np.nan, v)
    return sign * v


#: The 127 non-negative finite E4M3 values in code order 0x00..0x7E
#: (ascending, so the index of a value is its code).
E4M3_POSITIVE_TABLE = e4m3_decode(np.arange(0x7F))


def _round_to_table_rne(v: np.ndarray, table: np.ndarray) -> np.ndarray:
    """Index of the nearest entry of the ascending ``table`` to each
    non-negative ``v``; a tie goes to the even index; values at or beyond the
    last entry take the last index (saturation).  Comparisons are exact:
    ``v`` is float32 and the table and its midpoints are exact in float64."""
    v = np.asarray(v, dtype=np.float64)
    last = len(table) - 1
    lo = np.searchsorted(table, v, side="right") - 1
    lo = np.clip(lo, 0, last)
    hi = np.minimum(lo + 1, last)
    mid = (table[lo] + table[hi]) / 2.0
    pick_hi = (v > mid) | ((v == mid) & (hi % 2 == 0))
    idx = np.where(pick_hi, hi, lo)
    return np.where(v >= table[last], last, idx)


def e4m3_encode_rne_sat(s_f) -> np.ndarray:
    """E4M3 code of non-negative float32 ``s_f`` under reading R3: nearest
    E4M3 value, tie to the even code, saturating at 448 (0x7E)."""
    s = np.asarray(s_f, dtype=np.float32)
    if np.any(s < 0) or np.any(np.isnan(s)):
        raise ValueError("E4M3 scale encode expects non-negative finite input")
    return _round_to_table_rne(s, E4M3_POSITIVE_TABLE).astype(np.uint8)


def e2m1_encode_rne_sat(y, sign_source=None) -> np.ndarray:
    """4-bit E2M1 code of float32 ``y`` under reading R3: nearest magnitude in
    {0, .5, 1, 1.5, 2, 3, 4, 6}, tie to the even code, saturating at 6; bit 3
    is the sign bit of ``sign_source`` (default ``y``), kept on zero."""
    y = np.asarray(y, dtype=np.float32)
    src = y if sign_source is None else np.asarray(sign_source, dtype=np.float32)
    mag_code = _round_to_table_rne(np.abs(y), E2M1_MAGNITUDES).astype(np.uint8)
    return mag_code | (np.signbit(src).astype(np.uint8) << 3)


def e8m0_decode(codes) -> np.ndarray:
    """Value of E8M0 bytes (MXFP4 block scale, Preliminaries): 2^(e-127),
    0xFF is NaN."""
    e = np.asarray(codes, dtype=np.int64)
    v = np.exp2(e.astype(np.float64) - 127.0)
    return np.where(e == 255, np.nan, v)


# ---------------------------------------------------------------------------
# BF16 helpers (inputs and outputs of the path are BF16 bit patterns)
# ---------------------------------------------------------------------------

def bf16_bits_to_f32(bits) -> np.ndarray:
    """Exact widening of BF16 bit patterns (uint16) to float32."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def f64_to_bf16_bits_rne(v) -> np.ndarray:
    """Round float64 values to BF16 (nearest, ties to even) in one step.

    Done exactly with integer arithmetic on the float64 bit pattern (float64
    -> float32 -> bf16 would round twice).  Finite inputs only; magnitudes
    beyond the BF16 range become infinities."""
    v = np.atleast_1d(np.asarray(v, dtype=np.float64))
    if not np.all(np.isfinite(v)):
        raise ValueError("finite inputs only")
    sign = np.signbit(v).astype(np.uint32)
    a = np.abs(v)
    # a = m * 2^e, m in [0.5, 1) (exact).  BF16 keeps 8 significant bits, so
    # one ulp is 2^(e-8); below the normal range the grid is 2^-133.
    _, e = np.frexp(a)
    quantum_exp = np.maximum(e.astype(np.int64) - 8, -133)
    scaled = np.ldexp(a, -quantum_exp)             # exact (power-of-two scaling)
    fl = np.floor(scaled)
    frac = scaled - fl
    q = fl + ((frac > 0.5) | ((frac == 0.5) & (np.fmod(fl, 2.0) == 1.0)))
    val = np.ldexp(q, quantum_exp)                 # rounded magnitude, exact
    with np.errstate(over="ignore"):
        f32 = val.astype(np.float32)               # exact unless it overflows
    bits = (f32.view(np.uint32) >> np.uint32(16)).astype(np.uint32)
    return (bits | (sign << np.uint32(15))).astype(np.uint16)


# ---------------------------------------------------------------------------
# NVFP4 quantizer (Preliminaries, Q(x) = S * Pi_FP4(x / S); readings R1-R5)
# ---------------------------------------------------------------------------

def pack_codes(codes4: np.ndarray) -> np.ndarray:
    """Reading R5: two 4-bit codes per byte, even element in the low nibble."""
    c = np.asarray(codes4, dtype=np.uint8)
    assert c.shape[-1] % 2 == 0
    return (c[..., 0::2] & 0xF) | ((c[..., 1::2] & 0xF) << 4)


def unpack_codes(packed: np.ndarray) -> np.ndarray:
    """Inverse of :func:`pack_codes`."""
    p = np.asarray(packed, dtype=np.uint8)
    out = np.empty(p.shape[:-1] + (p.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = p & 0xF
    out[..., 1::2] = p >> 4
    return out


def nvfp4_quantize_ref(x_bits: np.ndarray):
    """NVFP4 quantization of a BF16 matrix ``x_bits`` ([rows, K] uint16).

    Follows Preliminaries (16-element blocks, E4M3 block scale, E2M1
    elements, Q(x) = S * Pi_FP4(x / S)) with the FP32 operation order of
    reading R2, rounding of R3, zero handling of R4 and layout of R5.

    Returns ``(codes, scales, alpha)``: codes uint8 [rows, K/2], scales uint8
    [rows, K/16], alpha a numpy float32 scalar (the per-tensor decode scale).
    """
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    if x_bits.ndim != 2:
        raise ValueError("expects a 2-D [rows, K] array")
    rows, K = x_bits.shape
    if K % NVFP4_BLOCK:
        raise ValueError("K must be a multiple of 16")
    nb = K // NVFP4_BLOCK
    x = bf16_bits_to_f32(x_bits)
    absx = np.abs(x)
    sign = np.signbit(x).astype(np.uint8) << 3

    # step 1: per-tensor amax (exact)
    amax_g = np.float32(absx.max()) if x.size else np.float32(0.0)
    if amax_g == 0:
        # R4: all-zero tensor
        return (pack_codes(sign), np.zeros((rows, nb), np.uint8), np.float32(0.0))

    # step 2: per-tensor decode scale (R1, R2)
    alpha = np.float32(amax_g / ALPHA_DIVISOR)
    t = np.float32(alpha * np.float32(6.0))

    # step 3: per-block scale (Preliminaries: one E4M3 scale per 16 elements)
    xb = x.reshape(rows, nb, NVFP4_BLOCK)
    amax_b = np.abs(xb).max(axis=2)
    s_f = (amax_b / t).astype(np.float32)
    s_code = e4m3_encode_rne_sat(s_f)
    s_val = e4m3_decode(s_code).astype(np.float32)

    # step 4: element projection y = x / S computed as x * (1 / (s * alpha))
    d = (s_val * alpha).astype(np.float32)
    with np.errstate(divide="ignore"):
        r = (np.float32(1.0) / d).astype(np.float32)
    zero_block = s_code == 0
    r = np.where(zero_block, np.float32(0.0), r).astype(np.float32)
    y = (xb * r[:, :, None]).astype(np.float32)
    codes = e2m1_encode_rne_sat(y, sign_source=xb)
    codes = np.where(zero_block[:, :, None], sign.reshape(rows, nb, NVFP4_BLOCK), codes)
    return pack_codes(codes.reshape(rows, K)), s_code, alpha


def nvfp4_dequantize_ref(codes: np.ndarray, scales: np.ndarray, alpha) -> np.ndarray:
    """Decoded values alpha * s * q in float64 (exact: at most 2 + 4 + 24
    significant bits).  Reading R1."""
    q = e2m1_decode(unpack_codes(codes))
    rows, K = q.shape
    s = e4m3_decode(scales).reshape(rows, K // NVFP4_BLOCK, 1)
    qs = (q.reshape(rows, K // NVFP4_BLOCK, NVFP4_BLOCK) * s).reshape(rows, K)
    return np.float64(alpha) * qs


def nvfp4_unscaled_ref(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """s * q per element, float64 (exact), without the tensor scale."""
    q = e2m1_decode(unpack_codes(codes))
    rows, K = q.shape
    s = e4m3_decode(scales).reshape(rows, K // NVFP4_BLOCK, 1)
    return (q.reshape(rows, K // NVFP4_BLOCK, NVFP4_BLOCK) * s).reshape(rows, K)


# ---------------------------------------------------------------------------
# Block-scaled FP4 GEMM and the linear layer (Sec. 3.4 Stage 1, Sec. 4.1; R6)
# ---------------------------------------------------------------------------

def nvfp4_gemm_ref(a_codes, a_scales, a_alpha, b_codes, b_scales, b_alpha,
                   bias_bits=None) -> np.ndarray:
    """Exact-input GEMM of reading R6, returned in float64 before the BF16
    output rounding:  alpha_A alpha_B (A_qs @ B_qs^T) + bias.

    A is [M, K] (codes [M, K/2], scales [M, K/16]); B is [N, K].  The
    products (s q)(s q) carry at most 12 significant bits, so the float64
    matmul is exact up to its summation rounding (~1e-16 relative)."""
    aq = nvfp4_unscaled_ref(a_codes, a_scales)
    bq = nvfp4_unscaled_ref(b_codes, b_scales)
    acc = aq @ bq.T
    out = (np.float64(a_alpha) * np.float64(b_alpha)) * acc
    if bias_bits is not None:
        out = out + bf16_bits_to_f32(bias_bits).astype(np.float64)[None, :]
    return out


def nvfp4_linear_ref(x_bits, w_codes, w_scales, w_alpha, bias_bits=None):
    """The NVFP4 linear layer of the denoiser (Sec. 4.1, Stage 1 of Sec. 3.4):
    quantize the BF16 activations, then the block-scaled GEMM with the
    pre-quantized weights.  Returns ``(out_f64, (codes, scales, alpha))``."""
    xc, xs, xa = nvfp4_quantize_ref(x_bits)
    return nvfp4_gemm_ref(xc, xs, xa, w_codes, w_scales, w_alpha, bias_bits), (xc, xs, xa)


def bf16_output(out_f64) -> np.ndarray:
    """The BF16 rounding of R6's output (nearest, ties to even)."""
    return f64_to_bf16_bits_rne(out_f64)


# ---------------------------------------------------------------------------
# MXFP4 (Preliminaries: OCP MXFP4 = 32 elements under one E8M0 scale; RM1-RM3)
# ---------------------------------------------------------------------------

def mxfp4_quantize_ref(x_bits: np.ndarray):
    """MXFP4 quantization of a BF16 matrix ([rows, K], K % 32 == 0).

    Per 32-element block: E = floor(log2(max|x|)) - 2 (reading RM1, exact
    through frexp), the E8M0 byte E + 127 clamped to [0, 254] (0 for an
    all-zero block), and codes E2M1_RNE_SAT(x / 2^E) with the sign of x kept
    (RM2).  Returns ``(codes uint8 [rows, K/2], scales uint8 [rows, K/32])``.
    """
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    if x_bits.ndim != 2:
        raise ValueError("expects a 2-D [rows, K] array")
    rows, K = x_bits.shape
    if K % MXFP4_BLOCK:
        raise ValueError("K must be a multiple of 32")
    nb = K // MXFP4_BLOCK
    x = bf16_bits_to_f32(x_bits).astype(np.float64).reshape(rows, nb, MXFP4_BLOCK)
    amax = np.abs(x).max(axis=2) if x.size else np.zeros((rows, nb))
    _, e = np.frexp(np.where(amax > 0, amax, 1.0))       # amax = m 2^e, m in [0.5, 1)
    floor_log2 = e.astype(np.int64) - 1
    code = np.clip(floor_log2 - 2 + 127, 0, 254)
    code = np.where(amax > 0, code, 0).astype(np.int64)
    X = np.exp2((code - 127).astype(np.float64))
    y = x / X[:, :, None]                                # exact: power-of-two scaling
    y32 = y.astype(np.float32)
    # exact in binary32 wherever it matters: below the smallest normal (an
    # element some 2^149 under its block's amax) every value encodes to a
    # signed zero however it rounds
    normal = np.abs(y) >= 2.0 ** -126
    assert np.array_equal(y32.astype(np.float64)[normal], y[normal])
    q = e2m1_encode_rne_sat(y32, sign_source=x.astype(np.float32))
    return pack_codes(q.reshape(rows, K)), code.astype(np.uint8)


def mxfp4_unscaled_ref(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """X * q per element, float64 (exact)."""
    q = e2m1_decode(unpack_codes(codes))
    rows, K = q.shape
    X = e8m0_decode(scales).reshape(rows, K // MXFP4_BLOCK, 1)
    return (q.reshape(rows, K // MXFP4_BLOCK, MXFP4_BLOCK) * X).reshape(rows, K)


def mxfp4_gemm_ref(a_codes, a_scales, b_codes, b_scales, bias_bits=None) -> np.ndarray:
    """MXFP4 GEMM (RM3) in float64 before the BF16 output rounding: A [M, K],
    B [N, K].  Products X_A q_A X_B q_B are exact powers of two times at most
    4 significant bits; the float64 sum is exact up to summation rounding."""
    out = mxfp4_unscaled_ref(a_codes, a_scales) @ mxfp4_unscaled_ref(b_codes, b_scales).T
    if bias_bits is not None:
        out = out + bf16_bits_to_f32(bias_bits).astype(np.float64)[None, :]
    return out


def mxfp4_linear_ref(x_bits, w_codes, w_scales, bias_bits=None):
    """MXFP4 linear: quantize the activations, then the MXFP4 GEMM."""
    xc, xs = mxfp4_quantize_ref(x_bits)
    return mxfp4_gemm_ref(xc, xs, w_codes, w_scales, bias_bits), (xc, xs)
