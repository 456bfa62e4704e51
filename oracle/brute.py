"""Pure-Python brute force for tiny Q4NX problems -- TEST INFRASTRUCTURE ONLY.

A second, independent implementation of the oracle's definition, used to pin
the NumPy oracle on tiny shapes.  It uses no NumPy: bf16 values are decoded
from their bit fields into exact rationals, Eq. 3 is evaluated exactly and
rounded once to binary32 (round to nearest, ties to even, IEEE 754 signed-zero
rules), and the projection sums are exact rationals.  Bytes are read from the
blob one at a time at the offsets the block layout defines:

  block (i, j) at (i*KB + j)*5120; code (r, k) in byte 128r + k//2 of the
  block, low nibble for even k; scale / offset (r, c) at 4096 + 2(8r + c) and
  4608 + 2(8r + c), little-endian.
"""
from __future__ import annotations

import struct
from fractions import Fraction


def bf16_value(bits: int):
    """(sign, Fraction magnitude) of a finite bf16 bit pattern."""
    sign = (bits >> 15) & 1
    exp = (bits >> 7) & 0xFF
    man = bits & 0x7F
    if exp == 0xFF:
        raise ValueError("inf/nan is outside the format's domain")
    if exp == 0:
        mag = Fraction(man, 1) * Fraction(2) ** (-126 - 7)
    else:
        mag = Fraction(128 + man, 1) * Fraction(2) ** (exp - 127 - 7)
    return sign, mag


def round_to_f32(v: Fraction) -> Fraction:
    """Round an exact rational to the nearest binary32 value, ties to even."""
    if v == 0:
        return Fraction(0)
    neg = v < 0
    a = -v if neg else v
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    quantum = Fraction(2) ** (max(e, -126) - 23)
    n = a / quantum
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    r = fl * quantum
    if r >= Fraction(2) ** 128:
        raise OverflowError("outside binary32 range")
    return -r if neg else r


def f32_bits(sign: int, mag: Fraction) -> int:
    """binary32 bit pattern of an exactly representable value."""
    v = float(mag)  # exact: every binary32 value is a binary64 value
    b = struct.unpack("<I", struct.pack("<f", v))[0]
    return b | (sign << 31)


def eq3_bits(q: int, d_bits: int, m_bits: int) -> int:
    """float32 bit pattern of RN(d*q + m) with IEEE signed-zero rules."""
    ds, dm = bf16_value(d_bits)
    ms, mm = bf16_value(m_bits)
    d = -dm if ds else dm
    m = -mm if ms else mm
    prod = d * q
    prod_sign = ds  # q >= 0, so a zero product carries the sign of d
    exact = prod + m
    if exact == 0:
        if prod == 0 and m == 0:
            sign = 1 if (prod_sign and ms) else 0   # (-0) + (-0) = -0, else +0
        else:
            sign = 0                                 # x + (-x) = +0 under RN
        return sign << 31
    r = round_to_f32(exact)
    return f32_bits(1 if r < 0 else 0, abs(r))


def f32_from_bits(b: int) -> Fraction:
    v = struct.unpack("<f", struct.pack("<I", b))[0]
    return Fraction(v)


def read_code(blob, N: int, K: int, n: int, k: int) -> int:
    KB = -(-K // 256)
    i, r = divmod(n, 32)
    j, kk = divmod(k, 256)
    base = (i * KB + j) * 5120
    byte = blob[base + 128 * r + kk // 2]
    return (byte >> 4) & 0xF if kk % 2 else byte & 0xF


def read_group_value(blob, N: int, K: int, n: int, k: int, which: str) -> int:
    KB = -(-K // 256)
    i, r = divmod(n, 32)
    j, kk = divmod(k, 256)
    c = kk // 32
    base = (i * KB + j) * 5120 + (4096 if which == "scale" else 4608) + 2 * (8 * r + c)
    return blob[base] | (blob[base + 1] << 8)


def dequant_bits(blob, N: int, K: int):
    """list of lists of float32 bit patterns of the dequantized weights."""
    out = []
    for n in range(N):
        row = []
        for k in range(K):
            q = read_code(blob, N, K, n, k)
            d = read_group_value(blob, N, K, n, k, "scale")
            m = read_group_value(blob, N, K, n, k, "offset")
            row.append(eq3_bits(q, d, m))
        out.append(row)
    return out


def project_exact(blob, N: int, K: int, X_rows):
    """Exact rational Y[m][n] = sum_k x[m][k] * w[n][k] for bf16 rows X."""
    W = dequant_bits(blob, N, K)
    Wf = [[f32_from_bits(b) for b in row] for row in W]
    Y = []
    for xrow in X_rows:
        xv = []
        for b in xrow:
            s, mag = bf16_value(int(b))
            xv.append(-mag if s else mag)
        Y.append([sum((xv[k] * Wf[n][k] for k in range(K)), Fraction(0)) for n in range(N)])
    return Y


# ----------------------------------------------------------------------------
# quantizer (the reading of oracle.quantize, in exact rational arithmetic)
# ----------------------------------------------------------------------------
def round_sig(v: Fraction, bits: int) -> Fraction:
    """Round a nonzero rational of magnitude >= 2^-126 to `bits` significant
    bits, ties to even (the normal range of binary32 and bf16)."""
    neg = v < 0
    a = -v if neg else v
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    quantum = Fraction(2) ** (e - (bits - 1))
    n = a / quantum
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    r = fl * quantum
    return -r if neg else r


def bf16_bits_of(v: Fraction) -> int:
    """bf16 bit pattern of RNE_bf16(v) with magnitudes below 2^-100 flushed
    to a zero of the same sign (v a binary32 value)."""
    if v == 0 or abs(v) < Fraction(2) ** -101:
        return 0x8000 if v < 0 else 0
    r = round_sig(v, 8)
    if abs(r) < Fraction(2) ** -100:
        return 0x8000 if r < 0 else 0
    sign = 1 if r < 0 else 0
    a = abs(r)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    man = int(a / Fraction(2) ** e * 128) - 128
    return (sign << 15) | ((e + 127) << 7) | man


def quantize_group_exact(ws):
    """One group of float32 values (Python floats, already clamped) ->
    (codes, scale bits, offset bits), by exact arithmetic."""
    vals = [Fraction(w) for w in ws]
    lo, hi = min(vals), max(vals)
    diff = hi - lo
    d32 = round_to_f32(round_to_f32(diff) / 15) if diff != 0 else Fraction(0)
    s_bits = bf16_bits_of(d32)
    m_bits = bf16_bits_of(lo)  # a zero minimum is +0
    levels = [f32_from_bits(eq3_bits(q, s_bits, m_bits)) for q in range(16)]
    codes = []
    for v in vals:
        best, bq = None, 0
        for q in range(16):
            dist = abs(levels[q] - v)
            if best is None or dist < best:
                best, bq = dist, q
        codes.append(bq)
    return codes, s_bits, m_bits
