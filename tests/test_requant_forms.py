"""The kernels' fast forms of the dyadic requantization (Sec. 3.2.1, Eq. 1:
the scales are applied after the integer accumulation, as a dyadic multiply
and shift; rounding half up and saturation to [-127, 127] are the readings
this implementation takes), checked on the CPU against the integer
definition q = sat(floor((v * m + 2^(s-1)) / 2^s)).

* Linear epilogues.  Per channel, c = b m + 2^(s-1) folds the bias and the
  rounding into one 64-bit addend, and the accumulator is first clamped to
  [lo, hi] = [-L - b, L - b] saturated to int32, with L = floor(130 * 2^s /
  |m|) + 1 (past L the result saturates anyway; no clamp when L would exceed
  2^30):

      q = sat(int32((clamp(acc) * m + c) >> s))

  claimed exact for every shift in [1, 62], any multiplier and any bias with
  acc + b inside int32 (the method's int32 accumulator): no intermediate
  leaves int64 and the shifted value stays inside int32.
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

I32 = (-(1 << 31), (1 << 31) - 1)
I64 = (-(1 << 63), (1 << 63) - 1)


def rq_exact(acc, m, s):
    v = (acc * m + (1 << (s - 1))) >> s
    return max(-127, min(127, v))


def in_range(v, r):
    return r[0] <= v <= r[1]


# ------------------------------------------------------- linear epilogue form
def clamp_bounds(m, b, s, margin=130):
    """[lo, hi] for the accumulator; None when no clamp is needed."""
    L = 2 if m == 0 else (margin << s) // abs(m) + 1
    if L >= 1 << 30:
        return None
    return max(-L - b, I32[0]), min(L - b, I32[1])


def rq_linear(acc, b, m, s, margin=130):
    bounds = clamp_bounds(m, b, s, margin)
    a = acc if bounds is None else max(bounds[0], min(bounds[1], acc))
    c = b * m + (1 << (s - 1))
    assert in_range(c, I64), "addend overflow"
    x = a * m + c
    assert in_range(x, I64), "int64 overflow"
    v = x >> s                       # arithmetic shift: the floor
    assert in_range(v, I32), "int32 overflow"
    return max(-127, min(127, v))


def linear_cases(m, s, b, rng, n=300, kmax=1536):
    """Random accumulators over a K = 1536 int8 dot product (kept so that
    acc + b fits int32), the clamp edges and every rounding and saturation
    boundary of acc + b."""
    amax = kmax * 127 * 127
    lo_ok, hi_ok = max(-amax, I32[0] - b), min(amax, I32[1] - b)
    accs = set(int(a) for a in rng.integers(lo_ok, hi_ok + 1, n))
    accs.update({0, 1, -1, lo_ok, hi_ok})
    bounds = clamp_bounds(m, b, s)
    if bounds is not None:
        for e in bounds:
            accs.update({e - 1, e, e + 1})
    if m != 0:
        for q in list(range(-130, 131, 5)) + [-128, -127, 126, 127, 128]:
            t = Fraction((2 * q + 1) << s, 2 * m) - b  # acc + b at q + 1/2
            for a in (math.floor(t) - 1, math.floor(t), math.ceil(t), math.ceil(t) + 1):
                accs.add(a)
    return sorted(a for a in accs if lo_ok <= a <= hi_ok)


LIN_PARAMS = [(1, 13, 0), (3, 1, -5), (1 << 29, 30, 12345), (-(1 << 30), 31, -(1 << 20)),
              (12345, 20, 77), ((1 << 30) - 12345, 43, (1 << 21) - 1),
              (-((1 << 29) + 5), 40, -((1 << 21) - 1)), ((1 << 31) - 1, 43, 1 << 15),
              ((1 << 31) - 1, 36, -(1 << 15)), ((1 << 29) + 3, 38, 32768),
              ((1 << 31) - 1, 62, (1 << 31) - (1 << 25)), (1, 62, 5), (-3, 53, -(1 << 30)),
              ((1 << 31) - 1, 1, 7), (0, 17, 1 << 30), ((1 << 30) + 1, 50, -(1 << 31) + (1 << 25))]


@pytest.mark.parametrize("m,s,b", LIN_PARAMS)
@pytest.mark.parametrize("margin", [129, 130])
def test_linear_form_is_exact(m, s, b, margin):
    """Any clamp bound L in [129 * 2^s / |m| + 1, 2^30] works (the kernel's
    fp32 estimate of 130 * 2^s / |m| lies there)."""
    rng = np.random.default_rng(abs(m) % 1000 + s + margin)
    for acc in linear_cases(m, s, b, rng):
        assert rq_linear(acc, b, m, s, margin) == rq_exact(acc + b, m, s), (acc, b, m, s)


def test_linear_form_random_parameters():
    rng = np.random.default_rng(7)
    for _ in range(120):
        s = int(rng.integers(1, 63))
        m = int(rng.integers(-(1 << 31) + 1, 1 << 31))
        b = int(rng.integers(-(1 << 31) + 1, 1 << 31))
        for acc in linear_cases(m, s, b, rng, n=40):
            assert rq_linear(acc, b, m, s) == rq_exact(acc + b, m, s), (acc, b, m, s)


def test_linear_clamp_is_needed():
    """Without the clamp a small shift with a large multiplier leaves int32
    after the shift (m = 2^31 - 1, s = 1, acc = 2^24 gives about 2^54)."""
    m, s, acc = (1 << 31) - 1, 1, 1 << 24
    v = (acc * m + (1 << (s - 1))) >> s
    assert not in_range(v, I32)
    assert rq_linear(acc, 0, m, s) == rq_exact(acc, m, s) == 127


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
