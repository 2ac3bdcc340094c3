"""Exact-arithmetic references for the pins of the sign and TernGrad
aggregates, written with Python's fractions (no code shared with the
oracle or the HIP library).

The aggregate of those kinds is read as the sum that every order of exact
arithmetic reaches: NaN when a decoded value is NaN or when both infinities
occur, an infinity when one occurs, otherwise the exact rational sum of the
finite values rounded once to float32 (nearest, ties to even; an exact zero
gives +0.0; a sum at or beyond the overflow threshold gives an infinity).
"""
import math
from fractions import Fraction

import numpy as np

f32 = np.float32
_FLT_MAX = Fraction(float(np.finfo(np.float32).max))


def fraction_to_f32(q):
    """Round a rational to the nearest float32 (ties to even), with the
    float32 subnormal spacing 2^-149 and overflow to an infinity."""
    if q == 0:
        return f32(0.0)
    sign = -1 if q < 0 else 1
    q = abs(q)
    e = q.numerator.bit_length() - q.denominator.bit_length()
    if Fraction(2) ** e > q:
        e -= 1
    ex = max(e, -126) - 23            # weight of the last kept bit
    sc = q / Fraction(2) ** ex
    m = sc.numerator // sc.denominator
    rem = sc - m
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and m % 2 == 1):
        m += 1
    r = Fraction(m) * Fraction(2) ** ex
    if r > _FLT_MAX:                  # rounded past the largest finite value
        return f32(sign * np.inf)
    return f32(sign * float(r))


def exact_round_f32(values):
    """Exact rational sum of finite float32 values, rounded once."""
    return fraction_to_f32(sum((Fraction(float(v)) for v in values), Fraction(0)))


def xsum_f32(values):
    """The order-free aggregate sum of float32 values (see module text)."""
    vals = [float(v) for v in values]
    if any(math.isnan(v) for v in vals):
        return f32(np.nan)
    pinf = any(v == math.inf for v in vals)
    ninf = any(v == -math.inf for v in vals)
    if pinf and ninf:
        return f32(np.nan)
    if pinf:
        return f32(np.inf)
    if ninf:
        return f32(-np.inf)
    return exact_round_f32(vals)


def same_f32(a, b):
    """Bit equality of float32 values, any NaN equal to any NaN."""
    a = f32(a)
    b = f32(b)
    if np.isnan(a) or np.isnan(b):
        return bool(np.isnan(a) and np.isnan(b))
    return a.view(np.uint32) == b.view(np.uint32)


def same_f32_arrays(a, b):
    """Element-wise same_f32 over two float32 arrays."""
    a = np.ascontiguousarray(a, np.float32)
    b = np.ascontiguousarray(b, np.float32)
    if a.shape != b.shape:
        return False
    nan = np.isnan(a) | np.isnan(b)
    return bool(np.array_equal(np.isnan(a), np.isnan(b))
                and np.array_equal(a.view(np.uint32)[~nan], b.view(np.uint32)[~nan]))
