"""Exact-rational scalar re-implementation of the NVFP4 quantizer and GEMM,
used to pin the vectorized CPU oracle.

It shares nothing with the oracle: every value is a ``fractions.Fraction``,
IEEE-754 binary32 round-to-nearest-even is written out from its definition
(``rn32``), and the E4M3 / E2M1 value sets are enumerated from their bit-field
definitions (Preliminaries: E2M1 = 1 sign, 2 exponent, 1 mantissa bit; NVFP4 =
16 elements per E4M3 scale).  The FP32 operation order is reading R2 of the
oracle (per-tensor scale amax/2688, block scale amax_b/(6 alpha), elements
x * (1/(s alpha))).  Pure Python loops: small inputs only.
"""
from __future__ import annotations

from fractions import Fraction

F = Fraction


def _floor_log2(a: Fraction) -> int:
    """Largest e with 2^e <= a, for a > 0 (exact)."""
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while F(2) ** e > a:
        e -= 1
    while F(2) ** (e + 1) <= a:
        e += 1
    return e


def _round_half_even(v: Fraction) -> int:
    fl = v.numerator // v.denominator
    rem = v - fl
    if rem > F(1, 2) or (rem == F(1, 2) and fl % 2 == 1):
        return fl + 1
    return fl


def rn32(v: Fraction) -> Fraction:
    """Round a rational to the nearest IEEE-754 binary32 value, ties to even
    (24 significant bits, subnormal quantum 2^-149).  Overflow raises."""
    if v == 0:
        return F(0)
    sign = -1 if v < 0 else 1
    a = abs(v)
    e = max(_floor_log2(a), -126)
    quantum = F(2) ** (e - 23)
    r = _round_half_even(a / quantum) * quantum
    if r >= F(2) ** 128:
        raise OverflowError("binary32 overflow")
    return sign * r


def e2m1_values():
    """The 8 non-negative E2M1 magnitudes, from the bit fields: exponent field
    0 is subnormal (m * 1/2), else 2^(e-1) * (1 + m/2)."""
    vals = []
    for e in range(4):
        for m in range(2):
            vals.append(F(m, 2) if e == 0 else F(2) ** (e - 1) * (1 + F(m, 2)))
    return vals  # codes 0..7 in order


def e4m3_values():
    """The 127 non-negative finite E4M3 values, codes 0x00..0x7E: exponent
    field 0 subnormal (m/8 * 2^-6), else (1 + m/8) * 2^(e-7); field 15 with
    mantissa 7 is NaN and excluded."""
    vals = []
    for e in range(16):
        for m in range(8):
            if e == 15 and m == 7:
                continue
            vals.append(F(m, 8) * F(2) ** -6 if e == 0 else (1 + F(m, 8)) * F(2) ** (e - 7))
    return vals


E2M1 = e2m1_values()
E4M3 = e4m3_values()


def nearest_code(v: Fraction, table) -> int:
    """Code of the nearest table value to v >= 0: exact distance, tie to the
    even code, beyond the largest value saturates."""
    if v >= table[-1]:
        return len(table) - 1
    best = None
    for c, t in enumerate(table):
        dist = abs(v - t)
        if best is None or dist < best[0] or (dist == best[0] and c % 2 == 0):
            best = (dist, c)
    return best[1]


def bf16_bits_to_fraction(bits: int) -> Fraction:
    """Exact value of a BF16 bit pattern (finite only)."""
    s = (bits >> 15) & 1
    e = (bits >> 7) & 0xFF
    m = bits & 0x7F
    if e == 0xFF:
        raise ValueError("non-finite")
    v = F(m, 128) * F(2) ** -126 if e == 0 else (1 + F(m, 128)) * F(2) ** (e - 127)
    return -v if s else v


def quantize_exact(rows_bits):
    """rows_bits: list of rows of BF16 bit patterns (ints).  Returns (codes
    per row as lists of 4-bit ints, scale codes per row, alpha as Fraction)."""
    xs = [[bf16_bits_to_fraction(b) for b in row] for row in rows_bits]
    signs = [[(b >> 15) & 1 for b in row] for row in rows_bits]
    amax_g = max((abs(v) for row in xs for v in row), default=F(0))
    K = len(rows_bits[0]) if rows_bits else 0
    nb = K // 16
    if amax_g == 0:
        return ([[s << 3 for s in row] for row in signs], [[0] * nb for _ in xs], F(0))
    alpha = rn32(amax_g / 2688)
    t = rn32(alpha * 6)
    codes, scales = [], []
    for row, srow in zip(xs, signs):
        crow, scrow = [], []
        for b in range(nb):
            blk = row[16 * b:16 * b + 16]
            amax_b = max(abs(v) for v in blk)
            s_f = rn32(amax_b / t)
            sc = nearest_code(s_f, E4M3)
            scrow.append(sc)
            if sc == 0:
                crow.extend(s << 3 for s in srow[16 * b:16 * b + 16])
                continue
            d = rn32(E4M3[sc] * alpha)
            r = rn32(1 / d)
            for v, s in zip(blk, srow[16 * b:16 * b + 16]):
                y = rn32(v * r)
                crow.append((s << 3) | nearest_code(abs(y), E2M1))
        codes.append(crow)
        scales.append(scrow)
    return codes, scales, alpha


def decode_exact(code4: int, scale_code: int) -> Fraction:
    """s * q for one element (exact)."""
    q = E2M1[code4 & 7]
    q = -q if code4 & 8 else q
    return q * E4M3[scale_code]


def gemm_exact(a_codes, a_scales, a_alpha, b_codes, b_scales, b_alpha, bias=None):
    """Exact rational alpha_A alpha_B sum_k (s q)_A (s q)_B + bias[n];
    a_codes: [M][K] 4-bit codes, a_scales: [M][K/16]; B likewise [N][K]."""
    M, N = len(a_codes), len(b_codes)
    K = len(a_codes[0]) if M else 0
    out = []
    for m in range(M):
        row = []
        for n in range(N):
            acc = F(0)
            for k in range(K):
                acc += (decode_exact(a_codes[m][k], a_scales[m][k // 16])
                        * decode_exact(b_codes[n][k], b_scales[n][k // 16]))
            v = F(a_alpha) * F(b_alpha) * acc
            if bias is not None:
                v += bias[n]
            row.append(v)
        out.append(row)
    return out


def mx_quantize_exact(rows_bits):
    """MXFP4 by exact rationals: per 32-element block E = floor(log2 amax) - 2
    (the OCP MX rule), byte clamp(E + 127, 0, 254), 0 for an all-zero block,
    q = nearest E2M1 of x / 2^E (exact division by a power of two)."""
    codes, scales = [], []
    for row in rows_bits:
        xs = [bf16_bits_to_fraction(b) for b in row]
        crow, srow = [], []
        for b0 in range(0, len(row), 32):
            blk = xs[b0:b0 + 32]
            amax = max(abs(v) for v in blk)
            if amax == 0:
                sc = 0
            else:
                sc = min(max(_floor_log2(amax) - 2 + 127, 0), 254)
            srow.append(sc)
            X = F(2) ** (sc - 127)
            for v, bits in zip(blk, row[b0:b0 + 32]):
                crow.append((((bits >> 15) & 1) << 3) | nearest_code(abs(v / X), E2M1))
        codes.append(crow)
        scales.append(srow)
    return codes, scales


def mx_gemm_exact(a_codes, a_scales, b_codes, b_scales, bias=None):
    """Exact rational sum_k (X q)_A (X q)_B + bias[n]; codes [rows][K], scales
    [rows][K/32]."""
    def dec(c, s):
        q = E2M1[c & 7]
        return (-q if c & 8 else q) * F(2) ** (s - 127)
    out = []
    for m in range(len(a_codes)):
        row = []
        for n in range(len(b_codes)):
            acc = F(0)
            for k in range(len(a_codes[m])):
                acc += dec(a_codes[m][k], a_scales[m][k // 32]) * dec(b_codes[n][k], b_scales[n][k // 32])
            if bias is not None:
                acc += bias[n]
            row.append(acc)
        out.append(row)
    return out
