"""The attention kernel's FP64 form of the score requantization (Sec. 3.1's
dyadic requantization, round half up, saturated to [-127, 127]):

    q + 256 = clamp(trunc(fma(acc, m * 2^-s, 256.5)), 129, 383)

claimed exact for |acc| <= 2^20 (a 64-channel head of int8 products) and
s <= 43 when |acc * m / 2^s| + 257 stays below 2^31.  A fused multiply-add
rounds the exact value once; float() of an exact Fraction rounds the same
way (to nearest, ties to even), so this checks the formula on the CPU against
the integer definition, including exact ties and the saturation edges.
"""
from fractions import Fraction
import math

import numpy as np
import pytest


def rq_exact(acc, m, s):
    v = (acc * m + (1 << (s - 1))) >> s
    return max(-127, min(127, v))


def rq_fp64(acc, m, s):
    y = float(Fraction(acc * m, 1 << s) + Fraction(513, 2))  # one rounding
    return max(129, min(383, math.trunc(y))) - 256


def f64_ok(m, s):
    """The host's condition for taking the FP64 form."""
    return s <= 43 and ((abs(m) << 20) >> s) + 257 < (1 << 31)


def cases(m, s, rng, n=400):
    """Random accumulators plus every boundary of the rounding and of the
    saturation that fits |acc| <= 2^20."""
    accs = set(int(a) for a in rng.integers(-(1 << 20), (1 << 20) + 1, n))
    accs.update({0, 1, -1, 1 << 20, -(1 << 20)})
    if m != 0:
        for q in list(range(-130, 131, 7)) + [-128, -127, 126, 127, 128]:
            # accumulators whose value acc * m / 2^s sits at or next to q + 1/2
            t = Fraction((2 * q + 1) << s, 2 * m)
            for a in (math.floor(t) - 1, math.floor(t), math.ceil(t), math.ceil(t) + 1):
                if abs(a) <= 1 << 20:
                    accs.add(a)
    return sorted(accs)


# (m, s, whether unsaturated exact ties are among the cases)
PARAMS = [(1, 13, True), (3, 1, True), (1 << 29, 30, True), (-(1 << 30), 31, True),
          (12345, 20, False), ((1 << 30) - 12345, 43, False), (-((1 << 29) + 5), 40, False),
          ((1 << 20) + 7, 22, False), ((1 << 31) - 1, 43, False), ((1 << 31) - 1, 32, False)]


def tie_accs(m, s):
    """Accumulators with acc * m = 2^(s-1) mod 2^s (exact ties), for odd m."""
    if m % 2 == 0:
        return []
    a0 = ((1 << (s - 1)) * pow(m, -1, 1 << s)) % (1 << s)
    return [a for a in (a0, a0 - (1 << s), a0 + (1 << s), a0 - (2 << s))
            if abs(a) <= 1 << 20]


@pytest.mark.parametrize("m,s,has_ties", PARAMS)
def test_fp64_form_is_exact(m, s, has_ties):
    assert f64_ok(m, s)
    rng = np.random.default_rng(abs(m) % 1000 + s)
    ties = 0
    for acc in cases(m, s, rng) + tie_accs(m, s):
        assert rq_fp64(acc, m, s) == rq_exact(acc, m, s), (acc, m, s)
        v = Fraction(acc * m, 1 << s)
        ties += v.denominator == 2 and abs(v) < 127
    if has_ties:
        assert ties > 0


def test_random_parameters():
    rng = np.random.default_rng(7)
    n = 0
    while n < 60:
        s = int(rng.integers(1, 44))
        m = int(rng.integers(-(1 << 31) + 1, 1 << 31))
        if not f64_ok(m, s):
            continue
        n += 1
        for acc in cases(m, s, rng, n=50):
            assert rq_fp64(acc, m, s) == rq_exact(acc, m, s), (acc, m, s)


def test_bound_is_needed():
    """Past s = 43 one rounding can cross an integer.  At s = 51 an
    accumulator near 2^20 and m = floor((2^50 - 1) / acc) put acc * m / 2^51
    within 2^-45 below 1/2; 256.5 plus that rounds to 257 (the spacing of
    doubles there is 2^-44), while the exact result is 0.  The host sends
    such shifts to the integer path."""
    s = 51
    found = 0
    for acc in range((1 << 20) - 50000, (1 << 20) + 1):
        m = ((1 << (s - 1)) - 1) // acc
        gap = (1 << (s - 1)) - acc * m  # 2^(s-1) - acc * m, in [1, acc]
        if gap < 1 << (s - 45):
            assert not f64_ok(m, s)
            assert rq_exact(acc, m, s) == 0
            found += rq_fp64(acc, m, s) != 0
    assert found > 0
