"""The double-double arithmetic behind the device's cumulative gates, checked on
the CPU against exact rationals (the reading of Sec. 2's cumulative sum: c_i is
the float32 rounding of the exact prefix sum).

The steps below restate, in Python floats (IEEE float64), the pair arithmetic the
kernels use: TwoSum (Knuth) on the leading parts, a plain sum of the remainders,
TwoSum again; the float32 rounding of a pair, whose leading part decides unless it
is a float32 midpoint. The claims pinned here: for float32 addends whose partial
sums span at most 105 bits, the pair is the exact sum in any association, and its
float32 rounding is c; the span read from the pair sum of |x| is exact there."""
import math
import random
import struct
from fractions import Fraction

import numpy as np
import pytest

import oracle as orc

F32_MAX = 3.4028234663852886e38
F32_OVERFLOW = 3.4028235677973366e38      # the largest float32 plus half an ulp


def two_sum(a, b):
    s = a + b
    bb = s - a
    e = (a - (s - bb)) + (b - bb)
    return s, (e if math.isfinite(s) else 0.0)


def dd_add(a, b):
    s = two_sum(a[0], b[0])
    return two_sum(s[0], (a[1] + b[1]) + s[1])


def _f32_bits(x):
    return struct.unpack("<I", struct.pack("<f", x))[0]


def _f32_from_bits(b):
    return struct.unpack("<f", struct.pack("<I", b))[0]


def dd_to_f32(a):
    hi, lo = a
    with np.errstate(over="ignore"):
        r = float(np.float32(hi))
    if lo == 0.0:
        return r
    if math.isinf(r):
        if abs(hi) == F32_OVERFLOW and (lo < 0) == (hi > 0):
            return math.copysign(F32_MAX, hi)
        return r
    if hi == r:
        return r
    rb = _f32_bits(r)
    mag = rb & 0x7FFFFFFF
    other = _f32_from_bits((rb & 0x80000000) | (mag + 1 if abs(hi) > abs(r) else mag - 1))
    if hi == 0.5 * (r + other) and ((lo > 0) == (other > r)):
        r = other
    return r


def dd_top_exp(a):
    m, e = math.frexp(a[0])
    return e - 1 if (m == 0.5 and a[1] < 0) else e


def _exact_f32(fr):
    return float(orc.acp_oracle._fraction_to_f32(fr))


def _random_row(rng, n, lo_e, hi_e):
    xs = [float(np.float32(-math.ldexp(rng.random(), rng.randint(lo_e, hi_e)))) for _ in range(n)]
    if n > 1 and rng.random() < 0.3:
        xs[rng.randrange(n)] = float(np.float32(rng.random()))   # a positive gate too
    return xs


def test_rounding_of_a_pair_is_that_of_its_exact_value():
    """Pairs near float32 midpoints (on both sides, exactly on them, subnormal and
    near the overflow threshold) round like the exact value they hold."""
    rng = random.Random(11)
    for _ in range(20000):
        e = rng.randint(-140, 127)
        m = rng.randint(1 << 23, (1 << 24) - 1)
        ulp = Fraction(2) ** (e - 23)
        mid = Fraction(m) * ulp + ulp / 2
        k = rng.choice([0, 1, -1, rng.randint(-10**6, 10**6)])
        val = mid + k * ulp * Fraction(2) ** (-60 - rng.randint(0, 10))
        if rng.random() < 0.5:
            val = -val
        hi = float(val)
        lo = float(val - Fraction(hi))
        if Fraction(hi) + Fraction(lo) != val:
            continue                                  # not representable as a pair
        assert dd_to_f32((hi, lo)) == _exact_f32(val), val


@pytest.mark.parametrize("seed", range(6))
def test_pair_sums_are_exact_in_any_association_up_to_105_bits(seed):
    """Rows with spans from a few bits to beyond 105: summed in a random tree of
    pair additions, the pair equals the exact sum (and its leading part that sum's
    float64 rounding) whenever the span is at most 105 bits; the pair sum of |x|
    then reads the span exactly, and the float32 rounding of every running prefix
    is the oracle's c."""
    rng = random.Random(100 + seed)
    seen_wide = 0
    for _ in range(40):
        n = rng.randint(1, 200)
        xs = _random_row(rng, n, rng.randint(-110, 0), rng.randint(0, 40))
        arr = np.array(xs, dtype=np.float32)
        span = orc.cumsum_span_bits(arr)
        vals = [(x, 0.0) for x in xs]
        while len(vals) > 1:
            i = rng.randrange(len(vals) - 1)
            vals[i:i + 2] = [dd_add(vals[i], vals[i + 1])]
        exact = sum(Fraction(x) for x in xs)
        tot = vals[0]
        absd = (0.0, 0.0)
        for x in xs:
            absd = dd_add(absd, (abs(x), 0.0))
        run, cs = (0.0, 0.0), []
        for x in xs:
            run = dd_add(run, (x, 0.0))
            cs.append(dd_to_f32(run))
        if span > 105:
            # the rule: a wider span is read as at least 105 bits (flag bit 2)
            lsb = min(max(math.frexp(abs(x))[1] - 1, -126) - 23 for x in xs if x != 0)
            assert dd_top_exp(absd) - lsb >= 105, span
            continue
        seen_wide += span > 53
        assert Fraction(tot[0]) + Fraction(tot[1]) == exact and tot[0] == float(exact), span
        if any(xs):
            abs_exact = sum(Fraction(abs(x)) for x in xs)
            e_true = math.frexp(float(abs_exact))[1]
            if Fraction(2) ** (e_true - 1) > abs_exact:   # float rounding reached a power of two
                e_true -= 1
            assert dd_top_exp(absd) == e_true, span
        np.testing.assert_array_equal(np.array(cs, dtype=np.float32), orc.cumsum_exact_fraction(arr))
    assert seen_wide > 0


def test_pair_keeps_infinities_and_nans_like_a_float64_sum():
    """A non-finite gate keeps the low part at zero, so -inf, +inf and NaN travel
    through the leading part as through a float64 running sum."""
    run = (0.0, 0.0)
    for x, want in ((-1.5, -1.5), (-math.inf, -math.inf), (-2.0, -math.inf)):
        run = dd_add(run, (x, 0.0))
        assert run == (want, 0.0)
    run = dd_add(run, (math.inf, 0.0))
    assert math.isnan(run[0]) and run[1] == 0.0
