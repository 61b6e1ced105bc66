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
# IEEE binary16, OCP FP8 E5M2 (binary16-like), OCP FP8 E4M3 "FN": no
# infinity, the all-ones pattern is the only NaN, largest finite 448.
F16 = dict(p=11, emin=-14, emax=15, ebits=5, bias=15, total=16, qnan=0x7E00)
E5M2 = dict(p=3, emin=-14, emax=15, ebits=5, bias=15, total=8, qnan=0x7E)
E4M3 = dict(p=4, emin=-6, emax=8, ebits=4, bias=7, total=8, qnan=0x7F, fn=True)
NARROW = {"f16": F16, "e5m2": E5M2, "e4m3": E4M3}
CANON_NAN32 = 0x7FC00000
F64 = dict(p=53, emin=-1022, emax=1023, ebits=11, bias=1023, total=64)
CANON_NAN64 = 0x7FF8000000000000


def decode(bits: int, fmt=F32):
    """bits -> ("nan",) | ("inf", sign) | ("fin", sign, Fraction magnitude)."""
    mbits = fmt["p"] - 1
    s = (bits >> (fmt["total"] - 1)) & 1
    e = (bits >> mbits) & ((1 << fmt["ebits"]) - 1)
    m = bits & ((1 << mbits) - 1)
    if fmt.get("fn") and e == (1 << fmt["ebits"]) - 1:
        if m == (1 << mbits) - 1:
            return ("nan",)
    elif e == (1 << fmt["ebits"]) - 1:
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


def _fn_max(fmt) -> int:
    """Magnitude bits of the largest finite value of an "FN" format."""
    return (((1 << fmt["ebits"]) - 1) << (fmt["p"] - 1)) | ((1 << (fmt["p"] - 1)) - 2)


def f32_to_narrow(b: int, dtype: str) -> int:
    """Correctly rounded binary32 -> f16 / e5m2 / e4m3.  NaN keeps its sign and
    becomes the format's quiet NaN; e4m3 saturates at 448 (also for infinities)."""
    fmt = NARROW[dtype]
    sbit = ((b >> 31) & 1) << (fmt["total"] - 1)
    d = decode(b)
    if d[0] == "nan":
        return sbit | fmt["qnan"]
    if fmt.get("fn"):
        # every magnitude >= the largest finite value rounds to it or past it,
        # and past it saturates: the result is the largest finite value
        top = Fraction(2 * (1 << (fmt["p"] - 1)) - 2, 1 << (fmt["p"] - 1)) * Fraction(2) ** fmt["emax"]
        if d[0] == "inf" or d[2] >= top:
            return sbit | _fn_max(fmt)
        return encode_rounded(d[1], d[2], fmt)
    if d[0] == "inf":
        return sbit | (((1 << fmt["ebits"]) - 1) << (fmt["p"] - 1))
    return encode_rounded(d[1], d[2], fmt)


def narrow_to_f32(h: int, dtype: str) -> int:
    """Exact widening of f16 / e5m2 / e4m3 bits to binary32 bits."""
    d = decode(h, NARROW[dtype])
    if d[0] == "nan":
        return CANON_NAN32
    if d[0] == "inf":
        return (d[1] << 31) | 0x7F800000
    return encode_rounded(d[1], d[2], F32)


def div32(a: int, b: int) -> int:
    """Correctly rounded binary32 division a / b."""
    A, B = decode(a), decode(b)
    if A[0] == "nan" or B[0] == "nan":
        return CANON_NAN32
    s = A[1] ^ B[1]
    if A[0] == "inf":
        return CANON_NAN32 if B[0] == "inf" else (s << 31) | 0x7F800000
    if B[0] == "inf":
        return s << 31
    if B[2] == 0:
        return CANON_NAN32 if A[2] == 0 else (s << 31) | 0x7F800000
    return encode_rounded(s, A[2] / B[2])


def f32_bits_of_int(k: int) -> int:
    return encode_rounded(0 if k >= 0 else 1, Fraction(abs(k)))


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


def iop64(op: str, dtype: str, a: int, b: int) -> int:
    """64-bit integer op on uint64 bit patterns (sum/prod modulo 2^64)."""
    m = (1 << 64) - 1
    if op == "sum":
        return (a + b) & m
    if op == "prod":
        return (a * b) & m
    if dtype == "i64":
        sa = a - (1 << 64) if a >> 63 else a
        sb = b - (1 << 64) if b >> 63 else b
        r = max(sa, sb) if op == "max" else min(sa, sb)
        return r & m
    return max(a, b) if op == "max" else min(a, b)


# ---- binary64: the same exact-then-round construction at p = 53 --------
INF64 = 0x7FF0000000000000


def _sign_bits64(s: int) -> int:
    return s << 63


def add64(a: int, b: int) -> int:
    """Correctly rounded binary64 a + b (round to nearest even)."""
    A, B = decode(a, F64), decode(b, F64)
    if A[0] == "nan" or B[0] == "nan":
        return CANON_NAN64
    if A[0] == "inf" and B[0] == "inf":
        return CANON_NAN64 if A[1] != B[1] else a
    if A[0] == "inf":
        return a
    if B[0] == "inf":
        return b
    v = (-A[2] if A[1] else A[2]) + (-B[2] if B[1] else B[2])
    if v == 0:
        return _sign_bits64(1) if (A[1] and B[1]) else 0
    return encode_rounded(1 if v < 0 else 0, abs(v), F64)


def mul64(a: int, b: int) -> int:
    """Correctly rounded binary64 a * b."""
    A, B = decode(a, F64), decode(b, F64)
    if A[0] == "nan" or B[0] == "nan":
        return CANON_NAN64
    s = A[1] ^ B[1]
    if A[0] == "inf" or B[0] == "inf":
        other = B if A[0] == "inf" else A
        if other[0] == "fin" and other[2] == 0:
            return CANON_NAN64
        return _sign_bits64(s) | INF64
    return encode_rounded(s, A[2] * B[2], F64)


def div64(a: int, b: int) -> int:
    """Correctly rounded binary64 a / b."""
    A, B = decode(a, F64), decode(b, F64)
    if A[0] == "nan" or B[0] == "nan":
        return CANON_NAN64
    s = A[1] ^ B[1]
    if A[0] == "inf":
        return CANON_NAN64 if B[0] == "inf" else _sign_bits64(s) | INF64
    if B[0] == "inf":
        return _sign_bits64(s)
    if B[2] == 0:
        return CANON_NAN64 if A[2] == 0 else _sign_bits64(s) | INF64
    return encode_rounded(s, A[2] / B[2], F64)


def is_nan64(b: int) -> bool:
    return (b & INF64) == INF64 and (b & ((1 << 52) - 1)) != 0


def _order_key64(b: int):
    d = decode(b, F64)
    if d[0] == "inf":
        return (1 if d[1] == 0 else -1, 0, 0)
    v = -d[2] if d[1] else d[2]
    return (0, v, 0 if d[1] else 1)


def max64(a: int, b: int) -> int:
    if is_nan64(a) or is_nan64(b):
        return CANON_NAN64
    return a if _order_key64(a) >= _order_key64(b) else b


def min64(a: int, b: int) -> int:
    if is_nan64(a) or is_nan64(b):
        return CANON_NAN64
    return a if _order_key64(a) <= _order_key64(b) else b


FOPS64 = {"sum": add64, "prod": mul64, "max": max64, "min": min64}


def iop8(op: str, dtype: str, a: int, b: int) -> int:
    """8-bit integer op on byte values 0..255: sum/prod modulo 2^8, max/min
    signed for i8 and unsigned for u8 (computed on the bytes directly, not by
    widening)."""
    if op == "sum":
        return (a + b) & 0xFF
    if op == "prod":
        return (a * b) & 0xFF
    if dtype == "i8":
        sa = a - 256 if a & 0x80 else a
        sb = b - 256 if b & 0x80 else b
        r = max(sa, sb) if op == "max" else min(sa, sb)
        return r & 0xFF
    return max(a, b) if op == "max" else min(a, b)


FLOAT_DTYPES = ("f32", "bf16", "f16", "e4m3", "e5m2")


def reduce_column(vals_bits, dtype: str, op: str) -> int:
    """Left fold of one column of bit patterns; returns the output bit pattern.
    AVG: the SUM fold, then one binary32 division by the number of values."""
    if dtype in FLOAT_DTYPES:
        if dtype == "bf16":
            up, down = bf16_to_f32, f32_to_bf16
        elif dtype == "f32":
            up, down = (lambda x: x & 0xFFFFFFFF), (lambda x: x)
        else:
            up = lambda x: narrow_to_f32(x, dtype)          # noqa: E731
            down = lambda x: f32_to_narrow(x, dtype)        # noqa: E731
        fop = FOPS["sum" if op == "avg" else op]
        acc = up(vals_bits[0])
        for v in vals_bits[1:]:
            acc = fop(acc, up(v))
        if op == "avg":
            acc = div32(acc, f32_bits_of_int(len(vals_bits)))
        if op in ("max", "min") and is_nan32(acc):
            acc = CANON_NAN32      # a NaN among the values, whatever their number
        return down(acc)
    if dtype == "f64":
        fop = FOPS64["sum" if op == "avg" else op]
        acc = vals_bits[0]
        for v in vals_bits[1:]:
            acc = fop(acc, v)
        if op == "avg":
            acc = div64(acc, encode_rounded(0, Fraction(len(vals_bits)), F64))
        if op in ("max", "min") and is_nan64(acc):
            acc = CANON_NAN64
        return acc
    if dtype in ("i8", "u8"):
        acc = vals_bits[0] & 0xFF
        for v in vals_bits[1:]:
            acc = iop8(op, dtype, acc, v & 0xFF)
        return acc
    if dtype in ("i64", "u64"):
        m = (1 << 64) - 1
        acc = vals_bits[0] & m
        for v in vals_bits[1:]:
            acc = iop64(op, dtype, acc, v & m)
        return acc
    acc = vals_bits[0] & 0xFFFFFFFF
    for v in vals_bits[1:]:
        acc = iop(op, dtype, acc, v & 0xFFFFFFFF)
    return acc
