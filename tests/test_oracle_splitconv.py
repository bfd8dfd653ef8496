"""Pins of the oracle's scale-preserving split convolution (Sec. 3.2.2, Fig.
projector_split_conv) against what the paper and the mathematics fix:

* with every branch at the common scale (rescale factor exactly 1) the split
  convolution is the plain convolution of the concatenated feature maps;
* the branch rescale and the output requantization follow their definitions
  in exact rational arithmetic, ties included;
* against real-valued arithmetic with distinct branch scales the integer sum
  stays within the rounding bound of the dyadic rescales, so each branch is
  rescaled by its own factor;
* one branch reduces to a linear layer, branch order does not matter, and
  the bias enters at the common scale.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def rand_branches(g, M, N, chans):
    xs = [g.integers(-127, 128, (M, c)).astype(np.int8) for c in chans]
    ws = [g.integers(-127, 128, (N, c)).astype(np.int8) for c in chans]
    return xs, ws


def sat8(v):
    return max(-127, min(127, v))


def rq_exact(v, m, s):
    """floor(v * m / 2^s + 1/2) in exact rationals."""
    q = Fraction(v * m, 2 ** s) + Fraction(1, 2)
    return q.numerator // q.denominator


@pytest.mark.parametrize("chans", [(16,), (64, 64), (24, 40, 8), (192, 192, 192)])
def test_equal_scales_equal_concat_conv(chans):
    """Every branch rescale is exactly 1 (m / 2^s = 2^k / 2^k): the split
    convolution equals the convolution over the concatenated maps."""
    g = rng(sum(chans))
    M, N = 37, 48
    xs, ws = rand_branches(g, M, N, chans)
    k = [int(g.integers(1, 31)) for _ in chans]
    bm = [[1 << kk] for kk in k]
    bs = [[kk] for kk in k]
    bias = g.integers(-2 ** 15, 2 ** 15 + 1, N).astype(np.int32)
    om = g.integers(2 ** 29, 2 ** 30 + 1, N).astype(np.int32)
    os_ = g.integers(36, 42, N).astype(np.int32)
    got = oracle.split_conv(xs, ws, bm, bs, bias, om, os_)
    ref = oracle.linear(np.concatenate(xs, axis=1), np.concatenate(ws, axis=1), bias, om, os_)
    assert np.array_equal(got, ref)
    # and the pre-requant sum is the plain integer matmul
    A = oracle.split_conv_sum(xs, ws, bm, bs, bias)
    plain = np.concatenate(xs, 1).astype(np.int64) @ np.concatenate(ws, 1).T.astype(np.int64)
    assert np.array_equal(A, plain + bias)


@pytest.mark.parametrize("per_channel", [False, True])
def test_brute_force_exact_rationals(per_channel):
    g = rng(7 + per_channel)
    M, N, chans = 4, 5, (3, 6, 2)
    xs, ws = rand_branches(g, M, N, chans)
    nq = N if per_channel else 1
    bm, bs = [], []
    for b in range(len(chans)):
        bm.append(g.integers(1, 2 ** 31 - 1, nq).astype(np.int32))
        bs.append(g.integers(20, 40, nq).astype(np.int32))
    # a branch with rescale 1/2: odd partial sums are exact ties
    bm[1][:] = 1
    bs[1][:] = 1
    bias = g.integers(-2 ** 15, 2 ** 15 + 1, N).astype(np.int32)
    om = g.integers(2 ** 29, 2 ** 30 + 1, nq).astype(np.int32)
    os_ = g.integers(30, 37, nq).astype(np.int32)
    A = oracle.split_conv_sum(xs, ws, bm, bs, bias)
    y = oracle.split_conv(xs, ws, bm, bs, bias, om, os_)
    ties = 0
    for m in range(M):
        for n in range(N):
            q = 0 if nq == 1 else n
            tot = int(bias[n])
            for b in range(len(chans)):
                acc = sum(int(xs[b][m, k]) * int(ws[b][n, k]) for k in range(chans[b]))
                ties += b == 1 and acc % 2 != 0
                tot += rq_exact(acc, int(bm[b][q]), int(bs[b][q]))
            assert A[m, n] == tot
            assert y[m, n] == sat8(rq_exact(tot, int(om[q]), int(os_[q])))
    assert ties > 0


def test_dequantized_error_bound():
    """Real-valued check with distinct activation scales: the rescaled integer
    sum A (at the common scale S_c = max S_b) matches sum_b S_b * acc_b / S_c
    within the rounding of each dyadic rescale."""
    g = rng(11)
    M, N, chans = 64, 32, (192, 192, 192)
    xs, ws = rand_branches(g, M, N, chans)
    scales = [0.0123, 0.0471, 0.0088]  # activation scales of the three maps
    Sc = max(scales)
    s = 30
    bm = [[int(round(2 ** s * Sb / Sc))] for Sb in scales]
    bs = [[s]] * 3
    assert bm[1][0] == 2 ** s  # the largest scale is the common one: factor 1
    bias = g.integers(-2 ** 15, 2 ** 15 + 1, N).astype(np.int32)
    A = oracle.split_conv_sum(xs, ws, bm, bs, bias)
    accs = [x.astype(np.int64) @ w.T.astype(np.int64) for x, w in zip(xs, ws)]
    real = bias.astype(np.float64) + sum(a * (Sb / Sc) for a, Sb in zip(accs, scales))
    bound = sum(0.5 + np.abs(a) * abs(m[0] / 2 ** s - Sb / Sc)
                for a, m, Sb in zip(accs, bm, scales)) + 1e-6
    assert np.all(np.abs(A - real) <= bound)
    # swapping two branches' scales breaks the bound: the pin sees the pairing
    swapped = oracle.split_conv_sum(xs, ws, [bm[1], bm[0], bm[2]], bs, bias)
    assert np.any(np.abs(swapped - real) > bound)


def test_single_branch_is_linear():
    g = rng(3)
    xs, ws = rand_branches(g, 50, 64, (128,))
    bias = g.integers(-2 ** 15, 2 ** 15 + 1, 64).astype(np.int32)
    om = g.integers(2 ** 29, 2 ** 30 + 1, 64).astype(np.int32)
    os_ = g.integers(30, 39, 64).astype(np.int32)
    got = oracle.split_conv(xs, ws, [[1 << 30]], [[30]], bias, om, os_)
    assert np.array_equal(got, oracle.linear(xs[0], ws[0], bias, om, os_))


def test_branch_order_invariance():
    g = rng(5)
    xs, ws = rand_branches(g, 20, 16, (32, 64, 16))
    bm = [g.integers(2 ** 28, 2 ** 30, 16).astype(np.int32) for _ in range(3)]
    bs = [g.integers(29, 32, 16).astype(np.int32) for _ in range(3)]
    bias = g.integers(-999, 999, 16).astype(np.int32)
    om, os_ = [1 << 30], [36]
    a = oracle.split_conv(xs, ws, bm, bs, bias, om, os_)
    p = [2, 0, 1]
    b = oracle.split_conv([xs[i] for i in p], [ws[i] for i in p], [bm[i] for i in p],
                          [bs[i] for i in p], bias, om, os_)
    assert np.array_equal(a, b)


def test_bias_at_common_scale():
    """Zero activations leave exactly the bias, whatever the branch rescales."""
    g = rng(9)
    xs = [np.zeros((3, c), np.int8) for c in (16, 48)]
    ws = [g.integers(-127, 128, (8, c)).astype(np.int8) for c in (16, 48)]
    bias = g.integers(-2 ** 15, 2 ** 15 + 1, 8).astype(np.int32)
    A = oracle.split_conv_sum(xs, ws, [[12345], [2 ** 29]], [[20], [31]], bias)
    assert np.array_equal(A, np.broadcast_to(bias.astype(np.int64), (3, 8)))
