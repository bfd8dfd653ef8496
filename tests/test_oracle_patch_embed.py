"""Pins of the oracle's patch embedding (a P x P stride-P convolution, its
requantization, and the positional embedding add; Table mappability lists
the encoder's patch embedding as a convolution plus an add):

* the convolution against torch's conv2d on the CPU (float64 holds every
  integer accumulator exactly), which fixes the patch and channel indexing;
* the same accumulators against a numpy patchify (reshape and transpose)
  followed by a matrix product;
* a zero image leaves the requantized bias plus the positional embedding.
"""
import numpy as np
import torch

import oracle


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def requant(acc, mult, shift):
    """Exact half-up requantization with saturation, in Python integers."""
    v = (int(acc) * int(mult) + (1 << (int(shift) - 1))) >> int(shift)
    return max(-127, min(127, v))


def residual(a, b, ma, mb, s):
    v = (int(a) * ma + int(b) * mb + (1 << (s - 1))) >> s
    return max(-127, min(127, v))


def case(seed, B=2, C=3, H=48, W=32, P=16, D=32):
    g = rng(seed)
    img = g.integers(-127, 128, (B, C, H, W)).astype(np.int8)
    w = g.integers(-127, 128, (D, C * P * P)).astype(np.int8)
    bias = g.integers(-2 ** 15, 2 ** 15 + 1, D).astype(np.int32)
    mult = g.integers(2 ** 29, 2 ** 30 + 1, D).astype(np.int32)
    shift = g.integers(36, 42, D).astype(np.int32)
    T = (H // P) * (W // P)
    pos = g.integers(-127, 128, (T, D)).astype(np.int8)
    return img, w, bias, mult, shift, pos


def test_patch_embed_matches_torch_conv2d():
    img, w, bias, mult, shift, pos = case(1)
    B, C, H, W = img.shape
    D, P = w.shape[0], 16
    ma, mb, s = 1 << 30, (1 << 29) + 12345, 31
    got = oracle.patch_embed(img, w, bias, mult, shift, pos, ma, mb, s)
    acc = torch.nn.functional.conv2d(torch.from_numpy(img.astype(np.float64)),
                                     torch.from_numpy(w.astype(np.float64)).reshape(D, C, P, P),
                                     torch.from_numpy(bias.astype(np.float64)), stride=P)
    acc = acc.numpy().astype(np.int64)  # [B, D, gh, gw]
    gh, gw = H // P, W // P
    for b in range(B):
        for py in range(gh):
            for px in range(gw):
                t = py * gw + px
                for n in range(D):
                    v = requant(acc[b, n, py, px], mult[n], shift[n])
                    assert got[b, t, n] == residual(v, pos[t, n], ma, mb, s)


def test_patch_embed_matches_patchify_matmul():
    img, w, bias, mult, shift, pos = case(2, B=1, H=64, W=80, D=48)
    B, C, H, W = img.shape
    P = 16
    # zero positional multiplier and a unit branch: y = requant of the conv
    got = oracle.patch_embed(img, w, bias, mult, shift, pos, 1 << 30, 0, 30)
    patches = img.reshape(B, C, H // P, P, W // P, P).transpose(0, 2, 4, 1, 3, 5)
    patches = patches.reshape(B, (H // P) * (W // P), C * P * P).astype(np.int64)
    acc = patches @ w.T.astype(np.int64) + bias
    ref = np.vectorize(requant)(acc, mult[None, None, :], shift[None, None, :]).astype(np.int8)
    assert np.array_equal(got, ref)


def test_zero_image_leaves_bias_and_position():
    img, w, bias, mult, shift, pos = case(3, B=1)
    img[:] = 0
    ma, mb, s = (1 << 30) - 7, 1 << 29, 31
    got = oracle.patch_embed(img, w, bias, mult, shift, pos, ma, mb, s)
    T, D = pos.shape
    for t in range(T):
        for n in range(D):
            assert got[0, t, n] == residual(requant(bias[n], mult[n], shift[n]), pos[t, n],
                                            ma, mb, s)
