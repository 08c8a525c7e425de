"""CPU: the floor division the conv kernels' tile set-up uses instead of an
integer division (integer division on the GPU takes several quarter-rate
multiplies): q = trunc(fl32(x * fl32(1/d) + fl32(0.5/d))), one fused
multiply-add in fp32, must equal floor(x / d) for 0 <= x < 2^22 and d >= 1.

The fused multiply-add is emulated exactly: x * r is exact in fp64 (24-bit by
24-bit significands), adding h in fp64 is exact where the exponents allow and
the single rounding to fp32 follows; the random cases are checked against
exact rationals."""
from fractions import Fraction

import numpy as np


def _q(x, d):
    r = np.float64(np.float32(1.0) / np.float32(d))
    h = np.float64(np.float32(0.5) / np.float32(d))
    v = (np.asarray(x, dtype=np.float64) * r + h).astype(np.float32)
    return np.trunc(v).astype(np.int64)


def test_small_operands_exhaustive():
    x = np.arange(0, 4096, dtype=np.int64)
    for d in range(1, 1025):
        assert np.array_equal(_q(x, d), x // d), f"d={d}"


def _rn32(v):
    """A positive rational rounded to the nearest fp32 value (ties to even),
    as an exact rational."""
    e = v.numerator.bit_length() - v.denominator.bit_length()
    if Fraction(2) ** e > v:
        e -= 1
    scale = Fraction(2) ** (23 - e)
    m = v * scale
    lo = m.numerator // m.denominator
    rem = m - lo
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1):
        lo += 1
    return Fraction(lo) / scale


def test_rounding_helper():
    for v in (1.0, 3.0, 1.0 / 3.0, 1e-3, 12345.678, 2.0 ** -20 * 3):
        assert _rn32(Fraction(v)) == Fraction(float(np.float32(v)))


def test_large_operands_exact_rationals():
    rng = np.random.default_rng(7)
    for _ in range(3000):
        d = int(rng.integers(1, 1 << 16))
        x = int(rng.integers(1, 1 << 22))
        r = Fraction(float(np.float32(1.0) / np.float32(d)))
        h = Fraction(float(np.float32(0.5) / np.float32(d)))
        v = _rn32(Fraction(x) * r + h)  # the fused multiply-add: one rounding
        assert int(v) == x // d, (x, d)


def test_boundaries():
    # the largest quotient's neighbourhood and exact multiples, where a
    # rounding error would show first
    for d in (1, 2, 3, 7, 9, 17, 34, 255, 1023, 4097, 65535):
        xs = [k * d + e for k in ((1 << 22) // d - 1, (1 << 22) // d - 2, 1, 2) for e in (-1, 0, 1, d - 1)]
        xs = [x for x in xs if 0 <= x < (1 << 22)]
        assert np.array_equal(_q(xs, d), np.asarray(xs) // d), d
