"""Binary32 arithmetic emulated with exact rationals (test helper, independent of any FPU).

fma(a, b, c) computes a*b + c exactly as a Fraction and rounds it once to
binary32 (round to nearest, ties to even, gradual underflow, overflow to inf),
following the IEEE-754 definition of fusedMultiplyAdd.  Signed zeros follow
IEEE-754 section 6.3: an exact zero sum of opposite-signed operands is +0 in
round-to-nearest; a sum of two -0 is -0; an underflow keeps the sign.
"""
import math
from fractions import Fraction

_MIN_EXP = -126     # smallest normal exponent
_MANT = 23          # stored significand bits
_QUANT_SUB = Fraction(1, 2 ** 149)
_MAX = (2 - Fraction(1, 2 ** 23)) * Fraction(2) ** 127


def _round_mag(q: Fraction) -> Fraction:
    """Round q > 0 to the nearest binary32 magnitude, ties to even (may return 0 or inf marker None)."""
    e = q.numerator.bit_length() - q.denominator.bit_length()
    if Fraction(2) ** e > q:
        e -= 1
    # now 2^e <= q < 2^(e+1)
    quantum = _QUANT_SUB if e < _MIN_EXP else Fraction(2) ** (e - _MANT)
    t = q / quantum
    n = t.numerator // t.denominator
    rem = t - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    r = n * quantum
    # overflow: values at or above MAX + half an ulp round to infinity
    if r > _MAX:
        return None
    return r


def to_f32(q: Fraction, sign_if_zero: float = 1.0) -> float:
    if q == 0:
        return math.copysign(0.0, sign_if_zero)
    r = _round_mag(abs(q))
    s = -1.0 if q < 0 else 1.0
    if r is None:
        return s * math.inf
    if r == 0:
        return math.copysign(0.0, s)
    return s * float(r)


def fma(a: float, b: float, c: float) -> float:
    if any(math.isnan(v) or math.isinf(v) for v in (a, b, c)):
        raise ValueError("finite operands only")
    exact = Fraction(a) * Fraction(b) + Fraction(c)
    if exact == 0:
        prod_neg = (math.copysign(1.0, a) * math.copysign(1.0, b)) < 0
        prod_zero = a == 0 or b == 0
        if prod_zero and c == 0:
            return -0.0 if (prod_neg and math.copysign(1.0, c) < 0) else 0.0
        return 0.0
    return to_f32(exact)


def add(a: float, b: float) -> float:
    return fma(a, 1.0, b)


def bf16_to_float(bits: int) -> float:
    import struct
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def float_bits(v: float) -> int:
    import struct
    return struct.unpack("<I", struct.pack("<f", v))[0]
