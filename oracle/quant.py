"""Quantization rules (Sec. III, Eq. quant, and the power-of-two rule of
Sec. III-B), written with exact arithmetic.

Readings of points the paper leaves open:
  * rounding: the paper rounds "to the next integer value" without a
    tie-break; the oracle uses round half up, R(v) = floor(v + 1/2), for
    every rounding of the method (weight taps, input taps, output requant);
  * the scale is s = x_max / 2^(n-1) and the quantizer clamps to
    [-2^(n-1), 2^(n-1)-1]; for int8 the positive maximum therefore maps to
    128 and saturates to 127, while -x_max maps to -128 exactly;
  * the power-of-two scale is 2^ceil(log2 s); with s = a/128 this is the
    smallest integer e with a <= 128 * 2^e (``cexp``), computed exactly.
    A zero maximum gets e = 0.
  * n-bit quantization (Eq. quant with n = bits) uses s = a / 2^(n-1) and
    [-2^(n-1), 2^(n-1)-1]; the Winograd domain of the int8/10 variant
    (Sec. V) has n = 10, everything else n = 8.
"""
from fractions import Fraction

import numpy as np

QMIN = -128
QMAX = 127


def round_half_up(v):
    """R(v) = floor(v + 1/2) for an exact rational (Fraction or int)."""
    v = Fraction(v)
    return (2 * v.numerator + v.denominator) // (2 * v.denominator)


def clamp(q, lo=QMIN, hi=QMAX):
    return max(lo, min(hi, q))


def qrange(bits=8):
    """Integer range [-2^(bits-1), 2^(bits-1) - 1] of a bits-wide quantizer."""
    return -(1 << (bits - 1)), (1 << (bits - 1)) - 1


def quantize_exact(x, e, bits=8):
    """Eq. quant with the power-of-two scale 2^e: clamp(R(x / 2^e)) for an
    exact rational x and an integer e (any sign)."""
    return clamp(round_half_up(Fraction(x) / Fraction(2) ** e), *qrange(bits))


def cexp(a, bits=8):
    """Smallest integer e with a <= 2^(bits-1) * 2^e (128 * 2^e for int8),
    i.e. ceil(log2(a / 2^(bits-1))), for an exact non-negative rational a.
    cexp(0) = 0."""
    a = Fraction(a)
    if a < 0:
        raise ValueError("cexp of a negative value")
    if a == 0:
        return 0
    q = a / (1 << (bits - 1))
    # first guess from bit lengths, then correct exactly
    e = q.numerator.bit_length() - q.denominator.bit_length()
    while Fraction(2) ** e < q:
        e += 1
    while Fraction(2) ** (e - 1) >= q:
        e -= 1
    return e


def shift_round_int(v, e):
    """R(v / 2^e) for integer arrays and an integer shift e >= 0, as the
    integer formula floor((v + 2^(e-1)) / 2^e); e = 0 is the identity."""
    v = np.asarray(v, dtype=np.int64)
    if e < 0:
        raise ValueError("negative shift")
    if e == 0:
        return v.copy()
    return np.floor_divide(v + (np.int64(1) << np.int64(e - 1)), np.int64(1) << np.int64(e))


def clamp_int8(v):
    return np.clip(np.asarray(v, dtype=np.int64), QMIN, QMAX)


def clamp_bits(v, bits=8):
    lo, hi = qrange(bits)
    return np.clip(np.asarray(v, dtype=np.int64), lo, hi)
