"""Pins of the I-ViT baseline operators (the forms that the paper's
Constrained Shiftmax and SD-ShiftGELU replace) at tensor level, and of the
failure modes the paper describes for them.

* Shiftmax with a fixed division precision (eq. shiftmax_original): the
  factor floor((2^M - 1) / S_sum) is 0 once S_sum >= 2^M, and coarse just
  below, while the constrained form keeps the output budget (Sec. 3.3.2).
  With s_d = 0 the constrained form reduces to it whenever S_sum < 2^31.
* ShiftGELU shifted by the row maximum (Sec. 3.3.1): a row with no positive
  I_p is exactly SD-ShiftGELU; a row with a large maximum drives both
  exponentials to the ShiftExp clamp and loses the sigmoid.
"""
import math

import numpy as np
import pytest

import oracle


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def test_fixed_m_factor_collapses_at_2_31():
    """Four equal maxima at I0 = 8192: S_sum = 4 * 8192 * 2^16 = 2^31, so the
    fixed-M (M = 31) factor is 0 and every output is 0; the constrained form
    calibrates s_d and keeps the row sum near 2^7."""
    x = np.zeros((1, 4), np.int8)
    assert np.all(oracle.shiftmax_ivit_rows(x, 8192, M=31) == 0)
    c = oracle.shiftmax_rows(x, 8192)
    assert 120 <= int(c.sum()) <= 128
    assert np.all(c == c[0, 0])


def test_fixed_m_factor_is_coarse_below_2_31():
    """Three equal maxima at I0 = 8192: S_sum = 3 * 2^29, the factor is
    floor((2^31 - 1) / (3 * 2^29)) = 1, so each output is 2^29 >> 24 = 32 and
    a quarter of the probability mass is lost; the constrained form gives 42."""
    x = np.zeros((1, 3), np.int8)
    assert np.array_equal(oracle.shiftmax_ivit_rows(x, 8192, M=31), np.full((1, 3), 32))
    assert np.array_equal(oracle.shiftmax_rows(x, 8192), np.full((1, 3), 42, np.int8))


def test_constrained_sd0_reduces_to_fixed_m():
    """With s_d = 0 the constrained form is eq. shiftmax_original with M = 31
    whenever S_sum <= 2^31 - 1 (small I0 keeps every row below)."""
    g = rng(1)
    x = g.integers(-127, 128, (64, 400)).astype(np.int8)
    for I0 in (8, 16, 31):
        assert np.array_equal(oracle.shiftmax_rows(x, I0, s_d=0),
                              oracle.shiftmax_ivit_rows(x, I0, M=31))


@pytest.mark.parametrize("M", [8, 16, 24, 32])
def test_fixed_m_budget(M):
    """0 <= sum of a row's outputs <= 2^(k_out-1): the factor never exceeds
    (2^M - 1) / S_sum."""
    g = rng(M)
    x = g.integers(-127, 128, (32, 256)).astype(np.int8)
    y = oracle.shiftmax_ivit_rows(x, 24, M=M).astype(np.int64)
    assert y.min() >= 0 and np.all(y.sum(axis=1) <= 128)


def test_shiftgelu_row_without_positive_ip_is_sd():
    """If no I_p of the row is positive, the row maximum (clamped at 0) is 0
    and ShiftGELU equals SD-ShiftGELU element by element."""
    row = np.arange(-127, 1, dtype=np.int8).reshape(1, -1)
    for I0 in (8, 16, 64):
        assert np.array_equal(oracle.shiftgelu_ivit_rows(row, I0, 1 << 30, 37),
                              oracle.sdshiftgelu_tensor(row, I0, 1 << 30, 37))


def test_shiftgelu_large_row_maximum_loses_the_sigmoid():
    """With 127 in the row (max I_p = 212 at I0 = 16), positive inputs whose
    shifted argument I_p - 212 reaches the ShiftExp clamp (Alg. 1: I_e =
    I + I/2 - I/16 <= -k_inter * I0) get a = a' = I0, so their sigmoid factor
    is floor(floor((2^31 - 1) / (2 I0)) * I0 / 2^24) = 63, i.e. 1/2, whatever
    x; SD-ShiftGELU follows the sigmoid, and its worst error is 5x smaller."""
    I0, k_inter = 16, 16
    Ip = lambda v: v + v // 2 + v // 8 + v // 16
    Ie = lambda v: v + v // 2 - v // 16
    mx = Ip(127)
    clamped = [v for v in range(1, 128) if Ie(Ip(v) - mx) <= -k_inter * I0]
    assert clamped == list(range(1, 21))
    half = ((2 ** 31 - 1) // (2 * I0)) * I0 >> 24
    assert half == 63
    for v in clamped:
        assert oracle.ivit_shiftgelu(v, mx, I0) == v * half
        if v >= 10:  # the true sigmoid of 1.702 x / I0 is above 0.73 there
            assert oracle.sdshiftgelu(v, I0) >= v * (half + 30)
    ivit = np.array([oracle.ivit_shiftgelu(v, mx, I0) for v in range(1, 128)])
    sd = np.array([oracle.sdshiftgelu(v, I0) for v in range(1, 128)])
    ideal = np.array([v / (1 + math.exp(-1.702 * v / I0)) * 128 for v in range(1, 128)])
    assert np.abs(ivit - ideal).max() > 5 * np.abs(sd - ideal).max()
