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
