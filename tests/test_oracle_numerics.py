"""Pins of the oracle's numerics against facts fixed outside the oracle.

Sec. 3 "Precision": codes in [0, 2^bits - 1], b = min, s = (max-min)/(2^bits-1).
Sec. 3 "Rounding": nearest with ties to the even code; stochastic rounding picks
x- or x+ with E = x.  Philox4x32-10: Random123 known answers and rocRAND's
header implementation.  FP16: numpy's float16 conversion (round to nearest even).
"""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest

import oracle
from exact import dequant_exact

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---- P1: code ranges and the min/max end points ------------------------------------------
@pytest.mark.parametrize("bits", [8, 4, 2])
def test_codes_in_range_and_endpoints(bits):
    K = 2**bits - 1
    rng = np.random.default_rng(10 + bits)
    for _ in range(200):
        d = int(rng.choice([16, 32, 128]))
        x = (rng.standard_normal(d) * rng.choice([1e-3, 0.05, 3.0])).astype(np.float32)
        codes, s, b = oracle.quantize_row(x, bits)
        assert codes.min() >= 0 and codes.max() <= K
        assert b == x.min()
        assert s == np.float32(np.float32(x.max() - x.min()) / np.float32(K))
        # with FP32 (s,b) and nearest rounding the row minimum maps to 0 and the maximum to K
        assert codes[np.argmin(x)] == 0
        assert codes[np.argmax(x)] == K
        # FP16 (s,b): still in range, and s, b are FP16 values
        codes16, s16, b16 = oracle.quantize_row(x, bits, sb_fp16=True)
        assert codes16.min() >= 0 and codes16.max() <= K
        assert np.float32(np.float16(s16)) == s16 and np.float32(np.float16(b16)) == b16


def test_constant_row_gives_zero_codes():
    x = np.full(16, 0.0375, dtype=np.float32)
    codes, s, b = oracle.quantize_row(x, 8)
    assert s == 0 and b == np.float32(0.0375) and not codes.any()
    assert np.all(dequant_exact(codes, s, b) == x)


def test_negative_zero_minimum_stored_as_positive_zero():
    x = np.array([-0.0, 0.5, 0.25, 1.0] * 4, dtype=np.float32)
    _, _, b = oracle.quantize_row(x, 8)
    assert b == 0 and not np.signbit(b)


# ---- P2: ties go to the even code --------------------------------------------------------
def test_round_half_to_even_int8():
    # min 0 and max 255 make s = 1 and b = 0 exactly, so v = x
    x = np.array([0, 255, 2.5, 3.5, 0.5, 1.5, 254.5, 100.5, 7.25, 7.75, 128, 64.5, 1, 2, 3, 4], dtype=np.float32)
    codes, s, b = oracle.quantize_row(x, 8)
    assert s == 1 and b == 0
    assert list(codes) == [0, 255, 2, 4, 0, 2, 254, 100, 7, 8, 128, 64, 1, 2, 3, 4]


def test_round_half_to_even_int4():
    x = np.array([0, 15, 7.5, 6.5, 0.5, 1.5, 14.5, 13.5, 2.25, 2.75, 8, 9, 10, 11, 12, 3], dtype=np.float32)
    codes, s, b = oracle.quantize_row(x, 4)
    assert s == 1 and b == 0
    assert list(codes) == [0, 15, 8, 6, 0, 2, 14, 14, 2, 3, 8, 9, 10, 11, 12, 3]


# ---- P3: stochastic rounding ---------------------------------------------------------------
def test_stochastic_rounding_unbiased_and_neighbouring():
    # s = 1, b = 0: v_j = x_j exactly; columns hold fractions on and off the grid
    fr = [0.0, 0.5, 0.25, 0.75, 0.1, 0.9, 0.01, 0.99, 0.3, 0.6, 0.125, 0.875, 0.0, 0.0]
    x = np.array([0.0, 255.0] + [10 + f for f in fr], dtype=np.float32)
    M = 4000
    acc = np.zeros(x.size)
    for step in range(M):
        codes, s, b = oracle.quantize_row(x, 8, stochastic=True, seed=77, step=step, table=3, row=11)
        assert s == 1 and b == 0
        lo = np.floor(x).astype(int)
        assert np.all((codes == lo) | (codes == lo + 1))
        acc += codes
    mean = acc / M
    frac = x - np.floor(x)
    bound = 4 * np.sqrt(frac * (1 - frac) / M) + 2.0**-24
    assert np.all(np.abs(mean - x) <= bound + 1e-12), (mean - x, bound)
    on_grid = frac == 0
    assert np.all(mean[on_grid] == x[on_grid])


def test_stochastic_rounding_depends_on_key():
    x = (np.random.default_rng(0).random(128) * 0.1).astype(np.float32)
    a = oracle.quantize_row(x, 4, stochastic=True, seed=1, step=5, table=0, row=9)[0]
    b = oracle.quantize_row(x, 4, stochastic=True, seed=1, step=5, table=0, row=9)[0]
    c = oracle.quantize_row(x, 4, stochastic=True, seed=2, step=5, table=0, row=9)[0]
    e = oracle.quantize_row(x, 4, stochastic=True, seed=1, step=6, table=0, row=9)[0]
    f = oracle.quantize_row(x, 4, stochastic=True, seed=1, step=5, table=0, row=10)[0]
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c) and not np.array_equal(a, e) and not np.array_equal(a, f)


def test_uniform_chi_square():
    vals = np.array([oracle.uniform(5, 3, t, r, c) for t in range(2) for r in range(100) for c in range(64)])
    assert vals.min() >= 0 and vals.max() < 1
    assert np.all(vals * 2**24 == np.floor(vals * 2**24))
    h = np.histogram(vals, bins=32, range=(0, 1))[0]
    e = vals.size / 32
    chi2 = ((h - e) ** 2 / e).sum()
    assert chi2 < 70  # 31 dof; p ~ 1e-4


# ---- P4: FP16 conversion -------------------------------------------------------------------
def test_fp16_matches_numpy():
    rng = np.random.default_rng(3)
    vals = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(0.05),
        (rng.random(5000) * 2**-14).astype(np.float32),          # fp16 subnormal range
        (rng.random(2000) * 2**-24).astype(np.float32),          # around the smallest subnormal
        np.array([65504, 65519.99, 65520, 70000, 2**-25, 2**-24, 3 * 2**-26, 1 + 2**-11, 1 + 3 * 2**-11,
                  -0.0, 0.0, np.inf, -np.inf, 1e-40, 2**-14 - 2**-25], dtype=np.float32),
    ])
    # exact halfway points between consecutive fp16 values
    h = np.arange(0x0000, 0x7BFF, 7, dtype=np.uint16).view(np.float16).astype(np.float32)
    h2 = np.arange(0x0001, 0x7C00, 7, dtype=np.uint16).view(np.float16).astype(np.float32)
    vals = np.concatenate([vals, (h[: len(h2)] + h2[: len(h)]) / np.float32(2)])
    for v in vals:
        want = np.array([v], dtype=np.float32).astype(np.float16).view(np.uint16)[0]
        assert oracle.f32_to_f16_bits(float(v)) == int(want), (v, hex(int(want)))
        back = oracle.f16_bits_to_f32(int(want))
        assert np.float32(back) == np.float16(np.uint16(want).view(np.float16)).astype(np.float32) or np.isnan(back)


# ---- P15: Philox4x32-10 --------------------------------------------------------------------
def _kat():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            w = [int(x, 16) for x in line.split()]
            rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


def test_philox_known_answers():
    for ctr, key, want in _kat():
        assert list(oracle.philox4x32_10(ctr, key)) == want


_PROBE = r"""
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
#include <cstdlib>
struct Probe : rocrand_device::philox4x32_10_engine {
  static uint4 run(uint4 c, uint2 k) { Probe p; return p.ten_rounds(c, k); }
};
int main(int argc, char** argv) {
  unsigned n = (unsigned)atoi(argv[1]);
  unsigned s = 0x12345u;
  for (unsigned i = 0; i < n; ++i) {
    unsigned v[6];
    for (int j = 0; j < 6; ++j) { s = s * 1664525u + 1013904223u; v[j] = s ^ (s >> 13) * 2654435761u; }
    uint4 r = Probe::run(make_uint4(v[0], v[1], v[2], v[3]), make_uint2(v[4], v[5]));
    printf("%u %u %u %u %u %u %u %u %u %u\n", v[0], v[1], v[2], v[3], v[4], v[5], r.x, r.y, r.z, r.w);
  }
}
"""


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc not installed")
def test_philox_matches_rocrand_header():
    """rocRAND's header-only philox4x32_10 engine (a library routine), host side."""
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "p.cpp")
        exe = os.path.join(d, "p")
        open(src, "w").write(_PROBE)
        subprocess.check_call(["hipcc", "-x", "hip", "--offload-arch=gfx950", "-O1", src, "-o", exe],
                              stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
        out = subprocess.check_output([exe, "300"], text=True)
    for line in out.splitlines():
        w = [int(x) for x in line.split()]
        assert list(oracle.philox4x32_10(w[0:4], w[4:6])) == w[6:10]


# ---- P14: requantizing a dequantized row is a fixed point -----------------------------------
@pytest.mark.parametrize("bits", [8, 4])
def test_requantize_idempotent_fp32_sb(bits):
    rng = np.random.default_rng(bits)
    for _ in range(100):
        x = (rng.random(128).astype(np.float32) * np.float32(0.1) - np.float32(0.05)).astype(np.float32)
        c1, s1, b1 = oracle.quantize_row(x, bits)
        y = dequant_exact(c1, s1, b1)
        c2, s2, b2 = oracle.quantize_row(y, bits)
        assert np.array_equal(c1, c2)
        assert b2 == b1
        assert abs(float(s2) - float(s1)) <= float(np.spacing(np.float32(s1)))


@pytest.mark.parametrize("bits", [8, 4])
def test_requantize_idempotent_fp16_sb(bits):
    rng = np.random.default_rng(100 + bits)
    for _ in range(100):
        x = (rng.random(64).astype(np.float32) * np.float32(0.1) - np.float32(0.05)).astype(np.float32)
        c1, s1, b1 = oracle.quantize_row(x, bits, sb_fp16=True)
        y = dequant_exact(c1, s1, b1)
        c2, s2, b2 = oracle.quantize_row(y, bits, sb_fp16=True)
        assert np.array_equal(c1, c2) and b2 == b1 and s2 == s1


# ---- P4b: FP16 table rounding (Sec. 3 "Rounding" with FP16 as the low precision) ------------
def _f16_samples(rng):
    return np.concatenate([
        rng.standard_normal(3000).astype(np.float32) * np.float32(0.05),
        (rng.random(800) * 2**-14).astype(np.float32) * rng.choice([-1, 1], 800).astype(np.float32),
        (rng.random(300) * 2**-23).astype(np.float32),
        rng.uniform(-65504, 65504, 300).astype(np.float32),
        np.array([0.0, -0.0, 1.0, -1.0, 65504.0, -65504.0, 65519.0, 65520.0, 7e4, -7e4, 2**-24, 2**-25,
                  3 * 2**-26, 1 + 2**-11, 1 + 3 * 2**-11, np.inf, -np.inf], dtype=np.float32),
    ])


def test_fp16_table_nearest_matches_numpy():
    from exact import f16_round_ref
    for x in _f16_samples(np.random.default_rng(21)):
        assert oracle.f16_round(float(x)) == f16_round_ref(x), x


def test_fp16_table_stochastic_threshold_is_exact():
    """x+ exactly when u < (x - x-)/(x+ - x-), checked at the uniforms straddling the
    threshold (the uniforms are multiples of 2^-24)."""
    from exact import f16_neighbours, f16_round_ref
    rng = np.random.default_rng(22)
    xs = [x for x in _f16_samples(rng) if np.isfinite(x)]
    for x in xs:
        us = [0.0, 1 - 2**-24, float(rng.random())]
        if abs(x) <= 65504:
            lo, hi = f16_neighbours(x)
            if lo != hi:
                p = (float(x) - float(lo)) / (float(hi) - float(lo))
                k = int(np.floor(p * 2**24))
                us += [(k - 1) * 2**-24, k * 2**-24, (k + 1) * 2**-24]
        for u in us:
            if 0 <= u < 1:
                got = oracle.f16_round(float(x), True, u)
                assert got == f16_round_ref(x, True, u), (x, u)
                if abs(x) <= 65504:
                    lo, hi = f16_neighbours(x)
                    assert got in (int(lo.view(np.uint16)), int(hi.view(np.uint16)))
    assert oracle.f16_round(7e4, True, 0.5) == 0x7BFF and oracle.f16_round(-7e4, True, 0.5) == 0xFBFF
    assert np.isnan(oracle.f16_bits_to_f32(oracle.f16_round(float("nan"), True, 0.5)))


def test_fp16_table_stochastic_unbiased():
    """Mean over draws of the pinned uniform equals x within 4 sigma (plus the 2^-24
    resolution of the uniform times the unit in the last place)."""
    xs = np.array([0.1, -0.3, 1 + 2**-12, 3e-6, -2.5e-7, 0.0375, 1000.3], dtype=np.float32)
    M = 3000
    from exact import f16_neighbours
    for i, x in enumerate(xs):
        vals = [oracle.f16_bits_to_f32(oracle.f16_round(float(x), True, oracle.uniform(9, k, 0, i, 0)))
                for k in range(M)]
        lo, hi = (float(v) for v in f16_neighbours(x))
        p = (float(x) - lo) / (hi - lo)
        sd = (hi - lo) * np.sqrt(p * (1 - p) / M)
        assert abs(np.mean(vals) - float(x)) <= 4 * sd + (hi - lo) * 2**-24, x
        assert set(vals) <= {lo, hi}


# ---- P1b/P2b: INT2 ---------------------------------------------------------------------------
def test_int2_codes_and_ties_to_even():
    x = np.array([0, 3, 0.5, 1.5, 2.5, 1, 2, 0.25, 0.75, 2.75, 1.25, 2.25, 3, 0, 1.75, 1.4], dtype=np.float32)
    codes, s, b = oracle.quantize_row(x, 2)
    assert s == 1 and b == 0
    assert list(codes) == [0, 3, 0, 2, 2, 1, 2, 0, 1, 3, 1, 2, 3, 0, 2, 1]


def test_int2_stochastic_rounding_unbiased():
    fr = [0.0, 0.5, 0.25, 0.75, 0.1, 0.9, 0.3, 0.6, 0.125, 0.875, 0.0, 0.0, 0.5, 0.2]
    x = np.array([0.0, 3.0] + [1 + f for f in fr], dtype=np.float32)
    M = 3000
    acc = np.zeros(x.size)
    for step in range(M):
        codes, s, b = oracle.quantize_row(x, 2, stochastic=True, seed=78, step=step, table=1, row=5)
        assert s == 1 and b == 0
        lo = np.floor(x).astype(int)
        assert np.all((codes == lo) | (codes == lo + 1))
        acc += codes
    frac = x - np.floor(x)
    bound = 4 * np.sqrt(frac * (1 - frac) / M) + 2.0**-24
    assert np.all(np.abs(acc / M - x) <= bound + 1e-12)
