"""The division-by-constant method the kernels use for set and key arithmetic
(Granlund and Montgomery, PLDI 1994): with l = ceil(log2 d) and
m = floor(2^32 (2^l - d)/d) + 1, n // d = (t + ((n - t) >> min(l, 1))) >> max(l - 1, 0)
where t = (m * n) >> 32.  Checked against exact integer division for divisors up to
2^31 - 1 (the largest table) at the numerators where an error would show first."""
import random


def magic(d):
    l = 0
    while l < 32 and (1 << l) < d:
        l += 1
    m = ((1 << 32) * ((1 << l) - d)) // d + 1
    return m, min(l, 1), max(l - 1, 0)


def div(n, c):
    m, s1, s2 = c
    t = (m * n) >> 32
    return (t + ((n - t) >> s1)) >> s2


def test_division_by_constant_is_exact():
    rnd = random.Random(7)
    divisors = (list(range(1, 1200)) + [3125, 1600, 62500, 2**30, 2**30 + 1, 2**31 - 1, 2**31 - 3, 641, 6700417]
                + [rnd.randrange(1, 2**31) for _ in range(1500)])
    base = [0, 1, 2, 2**31 - 1, 2**31, 2**32 - 2, 2**32 - 1] + [rnd.randrange(0, 2**32) for _ in range(100)]
    for d in divisors:
        c = magic(d)
        assert c[0] < 2**32  # fits the 32-bit multiplier
        top = (2**32 - 1) // d * d
        for n in base + [d - 1, d, d + 1, 2 * d - 1, 2 * d, top - 1, top]:
            if 0 <= n < 2**32:
                assert div(n, c) == n // d, (d, n)
