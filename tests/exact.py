"""Exact rational arithmetic rounded once to binary32 (test helper).

Used to state what a fused multiply-add or a dequantization must return without
going through any float pipeline: the exact value q*s + b is formed as a
Fraction and rounded to the nearest float32, ties to even.
"""
from fractions import Fraction

import numpy as np


def round_f32(q: Fraction) -> np.float32:
    if q == 0:
        return np.float32(0.0)
    neg = q < 0
    a = -q if neg else q
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    quantum_exp = max(e, -126) - 23
    m = a / (Fraction(2) ** quantum_exp)
    n = m.numerator // m.denominator
    rem = m - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    val = float(Fraction(n) * Fraction(2) ** quantum_exp)
    return np.float32(-val if neg else val)


def fma32(a, b, c) -> np.float32:
    return round_f32(Fraction(float(a)) * Fraction(float(b)) + Fraction(float(c)))


def dequant_exact(codes, scale, bias):
    """Row(s) of q*s+b, each element rounded once."""
    codes = np.asarray(codes)
    out = np.empty(codes.shape, dtype=np.float32)
    flat_c = codes.reshape(-1, codes.shape[-1]) if codes.ndim > 1 else codes.reshape(1, -1)
    s = np.atleast_1d(scale)
    b = np.atleast_1d(bias)
    o = out.reshape(flat_c.shape)
    cache = {}
    for i in range(flat_c.shape[0]):
        si, bi = float(s[i]), float(b[i])
        for j in range(flat_c.shape[1]):
            key = (int(flat_c[i, j]), si, bi)
            v = cache.get(key)
            if v is None:
                v = fma32(key[0], si, bi)
                cache[key] = v
            o[i, j] = v
    return out


def decode_rows(codes, scale, bias):
    """FP32 rows of exported low-precision rows: binary16 bit patterns (uint16 codes,
    an FP16 table) widen exactly; integer codes dequantize as q*s+b rounded once."""
    codes = np.asarray(codes)
    if codes.dtype == np.uint16:
        return codes.view(np.float16).astype(np.float32)
    return dequant_exact(codes, scale, bias)


def f16_neighbours(x):
    """(x-, x+): the consecutive binary16 values around float32 x, |x| <= 65504,
    from numpy's float16 type (equal when x is representable)."""
    h = np.float16(x)
    if float(h) == float(x):
        return h, h
    if float(h) > float(x):
        return np.nextafter(h, np.float16(-np.inf)), h
    return h, np.nextafter(h, np.float16(np.inf))


def f16_round_ref(x, stochastic=False, u=0.0):
    """binary16 bits of float32 x: numpy's nearest-even conversion, or stochastic
    rounding between the finite neighbours, x+ when u < (x - x-)/(x+ - x-) in exact
    rationals; beyond 65504 stochastic rounding saturates."""
    x = np.float32(x)
    if not stochastic or np.isnan(x):
        with np.errstate(over="ignore"):
            return int(np.float16(x).view(np.uint16))
    if x > 65504:
        return int(np.float16(65504).view(np.uint16))
    if x < -65504:
        return int(np.float16(-65504).view(np.uint16))
    lo, hi = f16_neighbours(x)
    if lo == hi:
        return int(lo.view(np.uint16))
    p = (Fraction(float(x)) - Fraction(float(lo))) / (Fraction(float(hi)) - Fraction(float(lo)))
    return int((hi if Fraction(float(u)) < p else lo).view(np.uint16))
