"""Brute-force reference for tiny inputs: exact rational arithmetic.

Independent of the oracle: every binary32 operation is computed exactly with
``fractions.Fraction`` and then rounded to the nearest representable value,
ties to even, by searching the quantum at the operand's binade.  This is the
IEEE 754 definition of a correctly rounded +, x and of the binary32 -> bf16
narrowing, written from the standard rather than from any implementation.

Values are passed around as bit patterns (Python ints).
"""
from __future__ import annotations

from fractions import Fraction

F32 = dict(p=24, emin=-126, emax=127, ebits=8, bias=127, total=32)
BF16 = dict(p=8, emin=-126, emax=127, ebits=8, bias=127, total=16)
CANON_NAN32 = 0x7FC00000


def decode(bits: int, fmt=F32):
    """bits -> ("nan",) | ("inf", sign) | ("fin", sign, Fraction magnitude)."""
    mbits = fmt["p"] - 1
    s = (bits >> (fmt["total"] - 1)) & 1
    e = (bits >> mbits) & ((1 << fmt["ebits"]) - 1)
    m = bits & ((1 << mbits) - 1)
    if e == (1 << fmt["ebits"]) - 1:
        return ("nan",) if m else ("inf", s)
    if e == 0:
        mag = Fraction(m) * Fraction(2) ** (fmt["emin"] - mbits)
    else:
        mag = Fraction(m | (1 << mbits)) * Fraction(2) ** (e - fmt["bias"] - mbits)
    return ("fin", s, mag)


def _floor_log2(q: Fraction) -> int:
    e = q.numerator.bit_length() - q.denominator.bit_length()
    # adjust so that 2^e <= q < 2^(e+1)
    while Fraction(2) ** e > q:
        e -= 1
    while Fraction(2) ** (e + 1) <= q:
        e += 1
    return e


def encode_rounded(sign: int, mag: Fraction, fmt=F32) -> int:
    """Round sign*mag to the nearest value of ``fmt`` (ties to even); return bits."""
    p, emin, emax = fmt["p"], fmt["emin"], fmt["emax"]
    mbits = p - 1
    sbit = sign << (fmt["total"] - 1)
    inf = sbit | (((1 << fmt["ebits"]) - 1) << mbits)
    if mag == 0:
        return sbit
    e = max(_floor_log2(mag), emin)
    quantum = Fraction(2) ** (e - mbits)
    q = mag / quantum
    n = q.numerator // q.denominator
    rem = q - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    if n == (1 << p):          # carried into the next binade
        n >>= 1
        e += 1
    if e > emax:
        return inf
    if n < (1 << mbits):       # subnormal (only possible at e == emin) or zero
        return sbit | n
    return sbit | ((e + fmt["bias"]) << mbits) | (n - (1 << mbits))


def add32(a: int, b: int) -> int:
    """Correctly rounded binary32 a + b (round to nearest even)."""
    A, B = decode(a), decode(b)
    if A[0] == "nan" or B[0] == "nan":
        return CANON_NAN32
    if A[0] == "inf" and B[0] == "inf":
        return CANON_NAN32 if A[1] != B[1] else a
    if A[0] == "inf":
        return a
    if B[0] == "inf":
        return b
    va = -A[2] if A[1] else A[2]
    vb = -B[2] if B[1] else B[2]
    v = va + vb
    if v == 0:
        # exact zero sum: -0 only when both operands are -0 (round to nearest)
        return 0x80000000 if (A[1] and B[1]) else 0
    return encode_rounded(1 if v < 0 else 0, abs(v))


def mul32(a: int, b: int) -> int:
    """Correctly rounded binary32 a * b."""
    A, B = decode(a), decode(b)
    if A[0] == "nan" or B[0] == "nan":
        return CANON_NAN32
    s = A[1] ^ B[1]
    if A[0] == "inf" or B[0] == "inf":
        other = B if A[0] == "inf" else A
        if other[0] == "fin" and other[2] == 0:
            return CANON_NAN32
        return (s << 31) | 0x7F800000
    return encode_rounded(s, A[2] * B[2])


def is_nan32(b: int) -> bool:
    return (b & 0x7F800000) == 0x7F800000 and (b & 0x7FFFFF) != 0


def _order_key(b: int):
    """Total order key for non-NaN binary32: value, then +0 above -0."""
    d = decode(b)
    if d[0] == "inf":
        return (1 if d[1] == 0 else -1, 0, 0)
    v = -d[2] if d[1] else d[2]
    return (0, v, 0 if d[1] else 1)


def max32(a: int, b: int) -> int:
    if is_nan32(a) or is_nan32(b):
        return CANON_NAN32
    return a if _order_key(a) >= _order_key(b) else b


def min32(a: int, b: int) -> int:
    if is_nan32(a) or is_nan32(b):
        return CANON_NAN32
    return a if _order_key(a) <= _order_key(b) else b


def f32_to_bf16(b: int) -> int:
    """Correctly rounded binary32 -> bf16; NaN keeps its sign and becomes 0x7FC0."""
    d = decode(b)
    if d[0] == "nan":
        return ((b >> 16) & 0x8000) | 0x7FC0
    if d[0] == "inf":
        return (d[1] << 15) | 0x7F80
    return encode_rounded(d[1], d[2], BF16)


def bf16_to_f32(h: int) -> int:
    return (h & 0xFFFF) << 16


FOPS = {"sum": add32, "prod": mul32, "max": max32, "min": min32}


def _s32(x: int) -> int:
    x &= 0xFFFFFFFF
    return x - (1 << 32) if x & 0x80000000 else x


def iop(op: str, dtype: str, a: int, b: int) -> int:
    """Integer op on uint32 bit patterns (sum/prod modulo 2^32)."""
    if op == "sum":
        return (a + b) & 0xFFFFFFFF
    if op == "prod":
        return (a * b) & 0xFFFFFFFF
    if dtype == "i32":
        sa, sb = _s32(a), _s32(b)
        r = max(sa, sb) if op == "max" else min(sa, sb)
        return r & 0xFFFFFFFF
    return max(a, b) if op == "max" else min(a, b)


def reduce_column(vals_bits, dtype: str, op: str) -> int:
    """Left fold of one column of bit patterns; returns the output bit pattern."""
    if dtype in ("f32", "bf16"):
        up = bf16_to_f32 if dtype == "bf16" else (lambda x: x & 0xFFFFFFFF)
        acc = up(vals_bits[0])
        for v in vals_bits[1:]:
            acc = FOPS[op](acc, up(v))
        if op in ("max", "min") and is_nan32(acc):
            acc = CANON_NAN32      # a NaN among the values, whatever their number
        return f32_to_bf16(acc) if dtype == "bf16" else acc
    acc = vals_bits[0] & 0xFFFFFFFF
    for v in vals_bits[1:]:
        acc = iop(op, dtype, acc, v & 0xFFFFFFFF)
    return acc
