"""The kernels' fast forms of the dyadic requantization (Sec. 3.1: round
half up, saturated to [-127, 127]), checked on the CPU against the integer
definition q = sat(floor((v * m + 2^(s-1)) / 2^s)).

* Linear epilogues, FP64 form.  Per channel, the accumulator is first
  clamped to [-L - b, L - b] with L = floor(130 * 2^s / |m|) + 1 (past L the
  result saturates anyway), then

      q + 256 = clamp(trunc(fma(acc, m 2^-s, c)), 129, 383),
      c = fma(b, m 2^-s, 256.5),

  claimed exact for s <= 43 and |b| < 2^21: c is representable, and the
  unsaturated values are multiples of 2^-s below 2^10.  A fused multiply-add
  rounds its exact value once; float() of an exact Fraction rounds the same
  way (to nearest, ties to even).
* Attention scores, 64-bit form, stored biased:

      q + 128 = clamp(int32((acc * m + 2^(s-1) + 128 * 2^s) >> s), 1, 255),

  for |acc| <= 2^20 (a 64-channel head).  The int64 value is exact for
  s <= 54; the host takes this form when the shifted value provably fits in
  int32 (any s >= 32; smaller s when |m| 2^20 / 2^s is small enough).
"""
from fractions import Fraction
import math

import numpy as np
import pytest


def rq_exact(acc, m, s):
    v = (acc * m + (1 << (s - 1))) >> s
    return max(-127, min(127, v))


# ------------------------------------------------------------------ FP64 form
def clamp_bound(m, s):
    """The accumulator bound: None when no clamp is needed (L >= 2^30)."""
    if m == 0:
        return 2
    L = (130 << s) // abs(m) + 1
    return None if L >= 1 << 30 else L


def rq_fp64(acc, b, m, s):
    L = clamp_bound(m, s)
    a = acc if L is None else max(-L - b, min(L - b, acc))
    scale = Fraction(m, 1 << s)            # a power-of-two scaling: exact
    c = float(b * scale + Fraction(513, 2))  # one rounding
    assert Fraction(c) == b * scale + Fraction(513, 2), "addend not representable"
    y = float(a * scale + Fraction(c))     # the fma: one rounding
    return max(129, min(383, math.trunc(y))) - 256


def f64_ok(b, s):
    return s <= 43 and abs(b) < 1 << 21


def fp64_cases(m, s, b, rng, n=300, kmax=1536):
    """Random accumulators over a K = 1536 int8 dot product, the clamp
    edges and every rounding and saturation boundary of acc + b."""
    amax = kmax * 127 * 127
    accs = set(int(a) for a in rng.integers(-amax, amax + 1, n))
    accs.update({0, 1, -1, amax, -amax})
    L = clamp_bound(m, s)
    if L is not None:
        for e in (-L - b, L - b):
            accs.update({e - 1, e, e + 1})
    if m != 0:
        for q in list(range(-130, 131, 5)) + [-128, -127, 126, 127, 128]:
            t = Fraction((2 * q + 1) << s, 2 * m) - b  # acc + b at q + 1/2
            for a in (math.floor(t) - 1, math.floor(t), math.ceil(t), math.ceil(t) + 1):
                if abs(a) <= amax:
                    accs.add(a)
    return sorted(accs)


LIN_PARAMS = [(1, 13, 0), (3, 1, -5), (1 << 29, 30, 12345), (-(1 << 30), 31, -(1 << 20)),
              (12345, 20, 77), ((1 << 30) - 12345, 43, (1 << 21) - 1),
              (-((1 << 29) + 5), 40, -((1 << 21) - 1)), ((1 << 31) - 1, 43, 1 << 15),
              ((1 << 31) - 1, 36, -(1 << 15)), ((1 << 29) + 3, 38, 32768)]


@pytest.mark.parametrize("m,s,b", LIN_PARAMS)
def test_linear_fp64_form_is_exact(m, s, b):
    assert f64_ok(b, s)
    rng = np.random.default_rng(abs(m) % 1000 + s)
    for acc in fp64_cases(m, s, b, rng):
        assert rq_fp64(acc, b, m, s) == rq_exact(acc + b, m, s), (acc, b, m, s)


def test_linear_fp64_random_parameters():
    rng = np.random.default_rng(7)
    for _ in range(60):
        s = int(rng.integers(1, 44))
        m = int(rng.integers(-(1 << 31) + 1, 1 << 31))
        b = int(rng.integers(-(1 << 21) + 1, 1 << 21))
        for acc in fp64_cases(m, s, b, rng, n=40):
            assert rq_fp64(acc, b, m, s) == rq_exact(acc + b, m, s), (acc, b, m, s)


def test_fp64_bound_is_needed():
    """Past s = 43 one rounding can cross an integer.  At s = 51 an
    accumulator near 2^20 and m = floor((2^50 - 1) / acc) put acc * m / 2^51
    within 2^-45 below 1/2; 256.5 plus that rounds to 257 (the spacing of
    doubles there is 2^-44), while the exact result is 0.  The host sends
    such shifts to the integer form."""
    s = 51
    found = 0
    for acc in range((1 << 20) - 50000, (1 << 20) + 1):
        m = ((1 << (s - 1)) - 1) // acc
        gap = (1 << (s - 1)) - acc * m  # 2^(s-1) - acc * m, in [1, acc]
        if gap < 1 << (s - 45):
            assert not f64_ok(0, s)
            assert rq_exact(acc, m, s) == 0
            y = float(Fraction(acc * m, 1 << s) + Fraction(513, 2))
            found += math.trunc(y) - 256 != 0
    assert found > 0


# ------------------------------------------------------------ 64-bit score form
def rq_score_fast(acc, m, s):
    x = acc * m + (1 << (s - 1)) + (128 << s)
    assert -(1 << 63) <= x < 1 << 63, "int64 overflow"
    v = x >> s                                     # arithmetic shift
    lo = ((v + (1 << 31)) % (1 << 32)) - (1 << 31)  # the low word as int32
    return max(1, min(255, lo)) - 128


def score_fast_ok(m, s):
    """The host's condition for the unclamped form."""
    return s <= 54 and (s >= 32 or ((abs(m) << 20) >> s) + 257 < 1 << 31)


def score_cases(m, s, rng, n=400):
    accs = set(int(a) for a in rng.integers(-(1 << 20), (1 << 20) + 1, n))
    accs.update({0, 1, -1, 1 << 20, -(1 << 20)})
    if m != 0:
        for q in list(range(-130, 131, 7)) + [-128, -127, 126, 127, 128]:
            t = Fraction((2 * q + 1) << s, 2 * m)
            for a in (math.floor(t) - 1, math.floor(t), math.ceil(t), math.ceil(t) + 1):
                if abs(a) <= 1 << 20:
                    accs.add(a)
    return sorted(accs)


SCORE_PARAMS = [(1, 13), (3, 1), (1 << 29, 30), ((1 << 30) + 1, 31), (-(1 << 30), 32),
                ((1 << 30) - 12345, 43), (-((1 << 29) + 5), 40), ((1 << 20) + 7, 22),
                ((1 << 31) - 1, 54), ((1 << 31) - 1, 32), (-((1 << 31) - 1), 33),
                ((1 << 10) - 1, 1)]


@pytest.mark.parametrize("m,s", SCORE_PARAMS)
def test_score_fast_form_is_exact(m, s):
    assert score_fast_ok(m, s)
    rng = np.random.default_rng(abs(m) % 997 + s)
    for acc in score_cases(m, s, rng):
        assert rq_score_fast(acc, m, s) == rq_exact(acc, m, s), (acc, m, s)


def test_score_fast_random_parameters():
    rng = np.random.default_rng(8)
    n = 0
    while n < 80:
        s = int(rng.integers(1, 55))
        m = int(rng.integers(-(1 << 31) + 1, 1 << 31))
        if not score_fast_ok(m, s):
            continue
        n += 1
        for acc in score_cases(m, s, rng, n=50):
            assert rq_score_fast(acc, m, s) == rq_exact(acc, m, s), (acc, m, s)


def test_score_fast_condition_is_needed():
    """Below s = 32 a large multiplier pushes the shifted value past int32:
    m = 2^30, s = 12 and acc = 2^20 give 2^38, whose low word is 0 (a
    wrong score of -128 before the clamp), so the host clamps the
    accumulator first; past s = 54 the int64 sum itself overflows."""
    assert not score_fast_ok(1 << 30, 12)
    assert rq_score_fast(1 << 20, 1 << 30, 12) != rq_exact(1 << 20, 1 << 30, 12)
    assert not score_fast_ok(1, 55)
    with pytest.raises(AssertionError, match="overflow"):
        rq_score_fast(1 << 20, (1 << 31) - 1, 56)
