"""GPU parity: every entry point of libilw.so against the CPU oracle on the
same seeded inputs, element by element.  Every operation is integer, so the
bar is bit-exact equality.

Sizes span several tiles with ragged tails, the edge cases of each operator
(empty inputs, single elements, constant rows, saturation, static and dynamic
s_d, in-place calls), and the five workloads at their full sizes: exactly
where the oracle finishes in seconds, on sampled images otherwise (with batch
independence checked on the GPU).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_24981_amd import ilw, synth

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

POISON = 0x5A


def _poison(t):
    if isinstance(t, torch.Tensor) and t.is_cuda and t.numel() > 0 and t.is_contiguous():
        t.reshape(-1).view(torch.uint8).fill_(POISON)
    return t


@pytest.fixture(autouse=True)
def poison_fresh_buffers(monkeypatch):
    """Every device buffer a test or the binding allocates (outputs and
    workspaces) starts filled with 0x5A, so an output element that a kernel
    never writes cannot pass by holding a stale, equal value left in the
    caching allocator by an earlier call."""
    empty, empty_like = torch.empty, torch.empty_like
    monkeypatch.setattr(torch, "empty", lambda *a, **k: _poison(empty(*a, **k)))
    monkeypatch.setattr(torch, "empty_like", lambda *a, **k: _poison(empty_like(*a, **k)))


def say(msg):
    print(f"[gpu] {msg}", flush=True)


def dev(a):
    return ilw.to_device(a)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_same(got, ref, what):
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    bad = np.flatnonzero(got.reshape(-1) != ref.reshape(-1))
    if bad.size:
        i = int(bad[0])
        raise AssertionError(f"{what}: {bad.size} of {ref.size} differ; first at flat "
                             f"{i}: got {got.reshape(-1)[i]} expected {ref.reshape(-1)[i]}")


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


# ------------------------------------------------------------------ linear
@pytest.mark.parametrize("M,N,K", [(1, 16, 16), (37, 48, 64), (300, 576, 192),
                                   (129, 768, 192), (257, 192, 768), (1000, 144, 208),
                                   (4099, 1152, 384),
                                   # K not a multiple of 64 on the other tiles: the
                                   # latency tile with 6 steps in flight, the one-wave
                                   # 64 x 64 tile and the 128 x 128 tile
                                   (500, 64, 400), (20000, 256, 208), (40000, 512, 208)])
@pytest.mark.parametrize("per_tensor", [False, True])
def test_linear(M, N, K, per_tensor):
    say(f"linear M={M} N={N} K={K} per_tensor={per_tensor}")
    g = rng(M * 7 + N + K)
    x = g.integers(-127, 128, (M, K)).astype(np.int8)
    w = g.integers(-127, 128, (N, K)).astype(np.int8)
    b = g.integers(-2 ** 15, 2 ** 15 + 1, N).astype(np.int32)
    nq = 1 if per_tensor else N
    mult = (g.integers(2 ** 29, 2 ** 30 + 1, nq) * g.choice([-1, 1], nq)).astype(np.int32)
    shift = g.integers(30, 44, nq).astype(np.int32)
    ref = oracle.linear(x, w, b, mult, shift)
    got = host(ilw.ilw_linear(dev(x), dev(w), dev(b), dev(mult), dev(shift)))
    assert_same(got, ref, "linear")


def _edge_channels(N, fallback):
    """Per-channel (mult, shift, bias) at the edges of the epilogue's
    requantization (shift 43, |bias| = 2^21 - 1, m = 0, odd m at shift 1:
    exact ties, tiny and huge scales); with extra, every 64-channel group also
    holds channels with shifts of 44, 50 and 62 and larger biases."""
    ms = [(1 << 31) - 1, -((1 << 31) - 1), 0, 1, 3, 1 << 29, -(1 << 30), 12345,
          (1 << 30) + 7, -5]
    ss = [43, 43, 30, 1, 1, 30, 31, 13, 40, 2]
    bs = [(1 << 21) - 1, -((1 << 21) - 1), 77, -3, 4, 1 << 20, -(1 << 20), 0, 12, -9]
    mult = np.array([ms[i % len(ms)] for i in range(N)], np.int32)
    shift = np.array([ss[i % len(ss)] for i in range(N)], np.int32)
    bias = np.array([bs[i % len(bs)] for i in range(N)], np.int32)
    if fallback:
        for g0 in range(0, N, 64):
            mult[g0 + 5], shift[g0 + 5], bias[g0 + 5] = (1 << 30) + 1, 50, 1 << 25
            mult[g0 + 17], shift[g0 + 17], bias[g0 + 17] = -(1 << 31) + 1, 44, -(1 << 21)
            mult[g0 + 40], shift[g0 + 40] = (1 << 31) - 1, 62
    return mult, shift, bias


@pytest.mark.parametrize("M", [300, 40000, 120000])  # 120000: more tiles than fit at once
@pytest.mark.parametrize("fallback", [False, True])
def test_linear_requant_forms(M, fallback):
    """The epilogue's requantization at its edges, including large shifts and
    biases, at a small-grid and a large-grid tile shape."""
    N, K = 256, 128
    say(f"linear requant forms M={M} fallback={fallback}")
    g = rng(M + fallback)
    x = g.integers(-127, 128, (M, K)).astype(np.int8)
    w = g.integers(-127, 128, (N, K)).astype(np.int8)
    mult, shift, bias = _edge_channels(N, fallback)
    ref = oracle.linear(x, w, bias, mult, shift)
    got = host(ilw.ilw_linear(dev(x), dev(w), dev(bias), dev(mult), dev(shift)))
    assert_same(got, ref, "linear requant forms")


def test_linear_no_bias_and_empty():
    say("linear without bias, M=0")
    g = rng(5)
    x = g.integers(-127, 128, (70, 96)).astype(np.int8)
    w = g.integers(-127, 128, (32, 96)).astype(np.int8)
    mult = np.full(1, 1 << 30, np.int32)
    shift = np.full(1, 40, np.int32)
    ref = oracle.linear(x, w, np.zeros(32, np.int32), mult, shift)
    got = host(ilw.ilw_linear(dev(x), dev(w), None, dev(mult), dev(shift)))
    assert_same(got, ref, "linear no bias")
    y = torch.full((0, 32), 5, dtype=torch.int8, device="cuda")
    ilw.ilw_linear(dev(x[:0]), dev(w), None, dev(mult), dev(shift), y=y)


# ------------------------------------------------------------------ Shiftmax
@pytest.mark.parametrize("rows,cols", [(1, 1), (7, 12), (33, 400), (10, 1600), (5, 4099),
                                       (3, 65536)])
@pytest.mark.parametrize("I0", [8, 64, 3000])
def test_shiftmax(rows, cols, I0):
    say(f"shiftmax rows={rows} cols={cols} I0={I0}")
    g = rng(rows * 131 + cols + I0)
    x = g.integers(-128, 128, (rows, cols)).astype(np.int8)
    x[0, :] = 7  # a constant row
    ref = oracle.shiftmax_rows(x, I0)
    got = host(ilw.ilw_shiftmax(dev(x), I0))
    assert_same(got, ref, "shiftmax dynamic")


@pytest.mark.parametrize("s_d,k_out,k_inter,m_p", [(0, 8, 16, 4), (3, 8, 16, 4),
                                                   (12, 8, 16, 4), (-1, 5, 16, 4),
                                                   (-1, 2, 16, 0), (-1, 8, 10, 7),
                                                   (20, 8, 16, 4)])
def test_shiftmax_params(s_d, k_out, k_inter, m_p):
    say(f"shiftmax s_d={s_d} k_out={k_out} k_inter={k_inter} m_p={m_p}")
    g = rng(77 + s_d + k_out)
    x = g.integers(-128, 128, (64, 400)).astype(np.int8)
    for I0 in (3, 16, 500):
        ref = oracle.shiftmax_rows(x, I0, k_inter, k_out, m_p, s_d)
        got = host(ilw.ilw_shiftmax(dev(x), I0, k_inter, k_out, m_p, s_d))
        assert_same(got, ref, f"shiftmax I0={I0}")


@pytest.mark.parametrize("rows,cols", [(16, 20), (8, 40), (8, 1100), (4, 5000)])
@pytest.mark.parametrize("m_p", [24, 31])
def test_shiftmax_large_m_p(rows, cols, m_p):
    """A large headroom m_p with I0 = 16383 (ShiftExp(0) near 2^30): the
    dynamic s_d = M_req + m_p - 31 reaches 35 to 44, so the output shift
    32 - k_out + s_d runs past 64 bits on the longer rows."""
    say(f"shiftmax large m_p={m_p} rows={rows} cols={cols}")
    g = rng(cols + m_p)
    x = g.integers(-128, 128, (rows, cols)).astype(np.int8)
    x[0, :] = 7
    ref = oracle.shiftmax_rows(x, 16383, m_p=m_p)
    got = host(ilw.ilw_shiftmax(dev(x), 16383, m_p=m_p))
    assert_same(got, ref, "shiftmax large m_p")


def test_shiftmax_in_place():
    say("shiftmax in place")
    x = synth.int8_tensor(9, (40, 333))
    ref = oracle.shiftmax_rows(x, 24)
    t = dev(x)
    ilw.ilw_shiftmax(t, 24, y=t)
    assert_same(host(t), ref, "shiftmax in place")


@pytest.mark.parametrize("rows,cols", [(5, 16), (9, 32), (17, 256), (33, 272), (6, 1024),
                                       (3, 2048), (1000, 1600), (4, 2064), (20001, 1024)])
@pytest.mark.parametrize("s_d", [-1, 0, 9])
def test_shiftmax_row_chunks(rows, cols, s_d):
    """Rows of whole 16-byte chunks held in registers (8, 32 or 64 lanes per
    row, partially filled lanes, several rows per wave, a row count that
    leaves the last wave's rows partly past the end), with the full int8
    range (-128 gives the 255-step table entry), static and dynamic s_d;
    2064 columns take the byte-wise kernel; 20 001 rows of 1024 make each
    wave of the largest grid walk more than one row (the next row's loads in
    flight)."""
    say(f"shiftmax row chunks rows={rows} cols={cols} s_d={s_d}")
    g = rng(rows * 7 + cols + s_d)
    x = g.integers(-128, 128, (rows, cols)).astype(np.int8)
    x[0, :] = -128
    x[0, 3] = 127
    if rows > 2:
        x[1, :] = 5
    for I0 in (8, 64, 4000):
        ref = oracle.shiftmax_rows(x, I0, s_d=s_d)
        got = host(ilw.ilw_shiftmax(dev(x), I0, s_d=s_d))
        assert_same(got, ref, f"shiftmax row chunks I0={I0}")
    t = dev(x)
    ilw.ilw_shiftmax(t, 30, s_d=s_d, y=t)
    assert_same(host(t), oracle.shiftmax_rows(x, 30, s_d=s_d), "shiftmax row chunks in place")


# ------------------------------------------------------------------ SD-ShiftGELU
@pytest.mark.parametrize("I0", [1, 8, 16, 37, 64, 1000, 16383])
def test_sdshiftgelu_exhaustive(I0):
    say(f"sdshiftgelu exhaustive I0={I0}")
    x = np.arange(-128, 128, dtype=np.int8)
    x = np.concatenate([x, x[::-1], x[:37]])  # 549 values: a ragged tail
    for m, s in ((1 << 30, 30), (1 << 30, 36), (-(1 << 29) - 7, 38), (1, 1)):
        ref = oracle.sdshiftgelu_tensor(x, I0, m, s)
        got = host(ilw.ilw_sdshiftgelu(dev(x), I0, m, s))
        assert_same(got, ref, f"gelu mult={m} shift={s}")
    for k_out, k_inter in ((2, 16), (5, 12), (8, 1)):
        ref = oracle.sdshiftgelu_tensor(x, I0, 1 << 30, 34, k_inter, k_out)
        got = host(ilw.ilw_sdshiftgelu(dev(x), I0, 1 << 30, 34, k_inter, k_out))
        assert_same(got, ref, f"gelu k_out={k_out} k_inter={k_inter}")


@pytest.mark.parametrize("n", [3_000_017, 70_000_003])
def test_sdshiftgelu_large_in_place(n):
    """In place; 70 000 003 elements make each thread of the largest grid
    walk its chunks more than once."""
    say(f"sdshiftgelu {n} elements in place")
    x = synth.int8_tensor(10, (n,), -128, 127)
    ref = oracle.sdshiftgelu_tensor(x, 21, 1 << 30, 36)
    t = dev(x)
    ilw.ilw_sdshiftgelu(t, 21, 1 << 30, 36, y=t)
    assert_same(host(t), ref, "gelu in place")


# ------------------------------------------------------------------ LayerNorm
@pytest.mark.parametrize("rows,C", [(1, 4), (7, 192), (100, 384), (3, 1028), (2, 16384)])
@pytest.mark.parametrize("iters", [10, 20])
@pytest.mark.parametrize("per_tensor", [False, True])
def test_layernorm(rows, C, iters, per_tensor):
    say(f"layernorm rows={rows} C={C} iters={iters} per_tensor={per_tensor}")
    g = rng(rows + C + iters)
    x = g.integers(-128, 128, (rows, C)).astype(np.int8)
    x[0, :] = -5                     # constant row: V = 0
    if rows > 2:
        x[1, :] = g.integers(-2, 3, C)  # tiny variance: Newton far from converged
    nq = 1 if per_tensor else C
    beta = g.integers(-2 ** 31, 2 ** 31, C).astype(np.int32)
    beta[: C // 2] >>= 5
    mult = (g.integers(2 ** 29, 2 ** 31, nq) * g.choice([-1, 1], nq)).astype(np.int32)
    shift = g.integers(44, 63, nq).astype(np.int32)
    ref = oracle.int_layernorm(x, beta, mult, shift, iters)
    got = host(ilw.ilw_int_layernorm(dev(x), dev(beta), dev(mult), dev(shift), iters))
    assert_same(got, ref, "layernorm")


@pytest.mark.parametrize("rows,C", [(8192, 192), (12345, 384), (9001, 48)])
@pytest.mark.parametrize("iters,per_tensor", [(10, False), (20, True)])
def test_layernorm_many_rows(rows, C, iters, per_tensor):
    """Many rows take the one-row-per-lane kernel (sum / sum of squares)."""
    say(f"layernorm many rows rows={rows} C={C} iters={iters} per_tensor={per_tensor}")
    g = rng(rows + C)
    x = g.integers(-128, 128, (rows, C)).astype(np.int8)
    x[::97] = 3                          # constant rows
    x[1::89] = g.integers(-1, 2, C)      # tiny variance
    nq = 1 if per_tensor else C
    beta = g.integers(-2 ** 31, 2 ** 31, C).astype(np.int32)
    beta[::2] >>= 6
    mult = (g.integers(2 ** 29, 2 ** 31, nq) * g.choice([-1, 1], nq)).astype(np.int32)
    shift = g.integers(44, 63, nq).astype(np.int32)
    ref = oracle.int_layernorm(x, beta, mult, shift, iters)
    t = dev(x)
    got = host(ilw.ilw_int_layernorm(t, dev(beta), dev(mult), dev(shift), iters, y=t))
    assert_same(got, ref, "layernorm many rows")


@pytest.mark.parametrize("rows,C", [(1, 16), (4097, 192), (5, 384), (12801, 384), (33, 1024),
                                    (9, 2048), (3000, 64)])
def test_layernorm_row_groups(rows, C):
    """The row kernel's lane groupings (4 lanes x 3 chunks up to 192
    channels, 8 x 3 up to 384, 16 x 4 up to 1024, 16 x 8 up to 2048), with
    several row groups per wave (the next group's loads in flight) and a
    last group partly past the end."""
    say(f"layernorm row groups rows={rows} C={C}")
    g = rng(rows * 3 + C)
    x = g.integers(-128, 128, (rows, C)).astype(np.int8)
    x[0, :] = 9
    beta = g.integers(-2 ** 26, 2 ** 26, C).astype(np.int32)
    mult = (g.integers(2 ** 29, 2 ** 30, C) * g.choice([-1, 1], C)).astype(np.int32)
    shift = g.integers(49, 52, C).astype(np.int32)
    for iters in (10, 20):
        ref = oracle.int_layernorm(x, beta, mult, shift, iters)
        got = host(ilw.ilw_int_layernorm(dev(x), dev(beta), dev(mult), dev(shift), iters))
        assert_same(got, ref, f"layernorm row groups iters={iters}")


def test_layernorm_in_place():
    say("layernorm in place")
    g = rng(12)
    x = g.integers(-128, 128, (333, 192)).astype(np.int8)
    beta = g.integers(-2 ** 26, 2 ** 26, 192).astype(np.int32)
    mult = g.integers(2 ** 29, 2 ** 30, 192).astype(np.int32)
    shift = g.integers(49, 52, 192).astype(np.int32)
    ref = oracle.int_layernorm(x, beta, mult, shift, 10)
    t = dev(x)
    ilw.ilw_int_layernorm(t, dev(beta), dev(mult), dev(shift), 10, y=t)
    assert_same(host(t), ref, "layernorm in place")


# ------------------------------------------------------------------ residual
@pytest.mark.parametrize("n", [1, 15, 16, 1000, 1_000_003, 40_000_017])
def test_residual(n):
    """Element-wise residual add; 40 000 017 elements make each thread of the
    largest grid walk its chunks more than once, with a ragged tail."""
    say(f"residual n={n}")
    g = rng(n)
    a = g.integers(-128, 128, n).astype(np.int8)
    b = g.integers(-128, 128, n).astype(np.int8)
    for ma, mb, s in ((1 << 30, 1 << 30, 31), (-(2 ** 31) + 1, 2 ** 31 - 1, 62), (3, -5, 1)):
        ref = oracle.residual_tensor(a, b, ma, mb, s)
        got = host(ilw.ilw_residual_add(dev(a), dev(b), ma, mb, s))
        assert_same(got, ref, f"residual {ma} {mb} {s}")


# ------------------------------------------------------------------ attention
ATTN_CASES = [
    # (B, grid_h, grid_w, win_h, win_w, heads)
    (1, 16, 16, 0, 0, 3),
    (2, 40, 40, 20, 20, 3),
    (1, 40, 40, 0, 0, 3),
    (2, 10, 10, 5, 5, 2),      # 25 tokens per window: ragged key/query blocks
    (1, 6, 10, 3, 5, 1),       # 15 tokens: fewer keys than one block
    (1, 1, 1, 0, 0, 1),        # a single token
    (1, 45, 45, 0, 0, 2),      # 2025 tokens: near the window limit
    (1, 32, 64, 0, 0, 2),      # 2048 tokens: the limit, a multiple of 64
    # 388 tokens (448 padded bytes, an exact fit of the Shiftmax words): only
    # the last two word steps masked, the first of them partly valid; 16-row
    # blocks (7 words over 16 lanes) and, at batch 40, 32-row blocks (14 over 8)
    (1, 4, 97, 0, 0, 1),
    (40, 4, 97, 0, 0, 1),
    # 300 tokens at 32-row blocks: 10 words over 8 lanes, an exact fit
    (26, 10, 30, 0, 0, 2),
]


@pytest.mark.parametrize("grid", [16, 4])
@pytest.mark.parametrize("I0", [1, 64, 16383])
@pytest.mark.parametrize("s_d", [20, 25, 31])
def test_attention_static_sd_small_denominator(s_d, I0, grid):
    """A static s_d far above the dynamic one: S_R = S_sum >> s_d is a few
    dozen or less, so F = floor((2^31 - 1) / S_R) is near 2^26..2^31, where an
    unrefined FP64 reciprocal is off by more than one unit (a regression
    case).  I0 at both ends of its range: with I0 = 1 and s_d >= 25 the
    shifted sum is 0 and clamps to 1 (F = 2^31 - 1); with I0 = 2^14 - 1 the
    exponentials use all of their 30 bits, and the 16-key rows (4 x 4 grid)
    keep the probabilities of nearly flat rows above one output unit.  Where
    every probability rounds to 0 (I0 = 1 with s_d >= 25; s_d = 31 unless
    I0 is large and the row short) the output is 0, a degenerate case the
    kernel must reproduce as well."""
    B, gh, gw, H = 1, grid, grid, 3
    say(f"attention static s_d={s_d}, I0={I0}, grid {grid}x{grid}")
    g = rng(900 + s_d + I0 + grid)
    D, T = 64 * H, gh * gw
    qkv = g.integers(-127, 128, (B, T, 3 * D)).astype(np.int8)
    p = {"score_mult": (1 << 29) + 4321, "score_shift": 39, "smax_I0": I0, "smax_s_d": s_d,
         "pv_mult": (1 << 29) + 777, "pv_shift": 36}
    ref = oracle.attention(qkv[0], gh, gw, 0, 0, H, 64, p["score_mult"], p["score_shift"],
                           p["smax_I0"], p["pv_mult"], p["pv_shift"], s_d=s_d)[None]
    got = host(ilw.ilw_attention(dev(qkv), gh, gw, 0, 0, H, p))
    assert_same(got, ref, "attention static s_d")


@pytest.mark.parametrize("case", ATTN_CASES)
@pytest.mark.parametrize("s_d", [-1, 4, 25])  # 25: output shifts of 32 and more
def test_attention(case, s_d):
    B, gh, gw, wh, ww, H = case
    say(f"attention B={B} grid={gh}x{gw} win={wh}x{ww} heads={H} s_d={s_d}")
    g = rng(gh * 100 + wh + H + s_d)
    D = 64 * H
    T = gh * gw
    qkv = g.integers(-127, 128, (B, T, 3 * D)).astype(np.int8)
    p = {"score_mult": int(g.integers(2 ** 29, 2 ** 30)), "score_shift": 39,
         "smax_I0": int(g.integers(8, 65)), "smax_s_d": s_d,
         "pv_mult": int(g.integers(2 ** 29, 2 ** 30)), "pv_shift": 36}
    ref = np.stack([oracle.attention(qkv[b], gh, gw, wh, ww, H, 64, p["score_mult"],
                                     p["score_shift"], p["smax_I0"], p["pv_mult"],
                                     p["pv_shift"], s_d=s_d) for b in range(B)])
    got = host(ilw.ilw_attention(dev(qkv), gh, gw, wh, ww, H, p))
    assert_same(got, ref, "attention")


@pytest.mark.parametrize("case", [
    # (B, grid_h, grid_w, win_h, win_w, heads, I0): one case per branch of the
    # kernel choice (row block, lanes and words per row, waves, 32- or 64-bit
    # lane sums, masking) not taken by the cases above; I0 = 3000 makes the
    # lane sums 64-bit
    (4, 32, 48, 0, 0, 3, 40),       # 1536 keys: 16-lane rows of 25 words, whole last step
    (4, 40, 40, 0, 0, 3, 3000),     # 1600 keys, 64-bit sums: 32 lanes x 13 words, split P V
    (1, 40, 40, 20, 20, 3, 3000),   # 400-key windows in 16-row blocks, 64-bit sums
    (4, 40, 40, 20, 20, 3, 3000),   # the same in 32-row blocks (8 lanes x 14 words)
    (1, 30, 30, 0, 0, 2, 40),       # 900 keys in 16-row blocks: 32 lanes x 8 words
    (2, 40, 40, 0, 0, 3, 40),       # 1600 keys in 16-row blocks: 64 lanes x 8 words
    (1, 34, 34, 0, 0, 2, 40),       # 1156 keys, 16 waves: 10 words
    (1, 42, 42, 0, 0, 2, 3000),     # 1764 keys, 16 waves: 14 words, 64-bit sums
])
def test_attention_dispatch(case):
    """Attention against the oracle on shapes that select kernel variants the
    other attention tests leave out."""
    B, gh, gw, wh, ww, H, I0 = case
    say(f"attention variants B={B} grid={gh}x{gw} win={wh}x{ww} heads={H} I0={I0}")
    g = rng(gh * 7 + gw + wh + H + I0)
    T, D = gh * gw, 64 * H
    qkv = g.integers(-127, 128, (B, T, 3 * D)).astype(np.int8)
    p = {"score_mult": int(g.integers(2 ** 29, 2 ** 30)), "score_shift": 39,
         "smax_I0": I0, "smax_s_d": -1,
         "pv_mult": int(g.integers(2 ** 29, 2 ** 30)), "pv_shift": 36}
    ref = np.stack([oracle.attention(qkv[b], gh, gw, wh, ww, H, 64, p["score_mult"],
                                     p["score_shift"], p["smax_I0"], p["pv_mult"],
                                     p["pv_shift"], s_d=-1) for b in range(B)])
    got = host(ilw.ilw_attention(dev(qkv), gh, gw, wh, ww, H, p))
    assert_same(got, ref, "attention variants")


@pytest.mark.parametrize("case", [
    # (B, grid_h, grid_w, heads, head_dim): grids of 32-row blocks large enough
    # for the split-key P V phase (rows past 1024 keys, 4 waves)
    (4, 40, 40, 3, 64),     # 1600 keys, 25 key blocks over 4 waves (7, 6, 6, 6)
    (4, 30, 50, 3, 64),     # 1500 keys: Shiftmax rows of 16 lanes, padded words
    (4, 37, 41, 3, 64),     # 1517 keys: the same with a ragged last word
    (5, 45, 45, 2, 64),     # 2025 keys: a ragged last block, 2048 padded
    (6, 26, 40, 3, 64),     # 1040 keys: 17 blocks, just past the threshold
    (4, 40, 40, 3, 32),     # 32-channel heads: two of the four groups unused
])
def test_attention_split_pv(case):
    B, gh, gw, H, hd = case
    say(f"attention split P V B={B} grid={gh}x{gw} heads={H} head_dim={hd}")
    g = rng(gh * 7 + gw + B + hd)
    D, T = hd * H, gh * gw
    qkv = g.integers(-127, 128, (B, T, 3 * D)).astype(np.int8)
    # scores spread over about 30 units of the int8 scale with a small I0:
    # peaked rows, so that Shiftmax leaves nonzero weights on 1000+ keys
    p = {"score_mult": int(g.integers(2 ** 29, 2 ** 30)), "score_shift": 40 if hd == 64 else 39,
         "smax_I0": int(g.integers(8, 17)), "smax_s_d": -1,
         "pv_mult": int(g.integers(2 ** 29, 2 ** 30)), "pv_shift": 34}
    ref = np.stack([oracle.attention(qkv[b], gh, gw, 0, 0, H, hd, p["score_mult"],
                                     p["score_shift"], p["smax_I0"], p["pv_mult"],
                                     p["pv_shift"]) for b in range(B)])
    got = host(ilw.ilw_attention(dev(qkv), gh, gw, 0, 0, H, p))
    assert_same(got, ref, "attention split P V")
    assert np.mean(ref == 0) < 0.1 and np.mean(np.abs(ref) == 127) < 0.5


# (score_mult, score_shift): the unclamped score form covers shifts 32..54,
# and smaller shifts when |acc * m / 2^s| stays inside int32 (|acc| <= 2^20);
# the rest clamp the accumulator first.
SCORE_RQ = [
    (1, 13),                      # unclamped: acc / 2^13, exact ties at acc = 4096 mod 8192
    ((1 << 30) - 12345, 43),      # unclamped, shift >= 32
    (-((1 << 29) + 5), 40),       # unclamped, negative scale
    ((1 << 20) + 7, 22),          # unclamped below 32, mostly saturated
    ((1 << 30) + 1, 31),          # unclamped at the largest shift below 32
    ((1 << 30) + 1, 44),          # unclamped
    ((1 << 31) - 1, 54),          # unclamped at its largest shift: every score rounds to 0
    ((1 << 31) - 1, 32),          # unclamped at shift 32, mostly saturated
    (-((1 << 31) - 1), 55),       # clamped: past 54
    ((1 << 31) - 1, 62),          # clamped at the largest shift
    (1 << 30, 12),                # clamped: the shifted value would overflow int32
]


@pytest.mark.parametrize("case", [(1, 40, 40, 0, 0, 1), (2, 10, 10, 5, 5, 2)])
@pytest.mark.parametrize("rqp", SCORE_RQ)
def test_attention_score_requant_paths(case, rqp):
    B, gh, gw, wh, ww, H = case
    sm, ss = rqp
    say(f"attention score rq m={sm} s={ss} B={B} grid={gh}x{gw} win={wh}x{ww} heads={H}")
    g = rng(ss * 7 + gh)
    D, T = 64 * H, gh * gw
    qkv = g.integers(-127, 128, (B, T, 3 * D)).astype(np.int8)
    p = {"score_mult": sm, "score_shift": ss, "smax_I0": int(g.integers(8, 65)),
         "smax_s_d": -1, "pv_mult": int(g.integers(2 ** 29, 2 ** 30)), "pv_shift": 36}
    ref = np.stack([oracle.attention(qkv[b], gh, gw, wh, ww, H, 64, sm, ss, p["smax_I0"],
                                     p["pv_mult"], p["pv_shift"]) for b in range(B)])
    got = host(ilw.ilw_attention(dev(qkv), gh, gw, wh, ww, H, p))
    assert_same(got, ref, "attention score requant")


@pytest.mark.parametrize("case", [(1, 1, 300, 0, 0, 8), (2, 6, 10, 3, 5, 4),
                                  (1, 15, 20, 0, 0, 2), (3, 1, 37, 0, 0, 1),
                                  (1, 40, 40, 0, 0, 2)])
def test_attention_head_dim_32(case):
    """32-channel heads (the decoder's self-attention: 300 queries, 8 heads)."""
    B, gh, gw, wh, ww, H = case
    say(f"attention hd32 B={B} grid={gh}x{gw} win={wh}x{ww} heads={H}")
    g = rng(gh * 31 + gw + H)
    D, T = 32 * H, gh * gw
    qkv = g.integers(-127, 128, (B, T, 3 * D)).astype(np.int8)
    p = {"score_mult": int(g.integers(2 ** 29, 2 ** 30)), "score_shift": 38,
         "smax_I0": int(g.integers(8, 65)), "smax_s_d": -1,
         "pv_mult": int(g.integers(2 ** 29, 2 ** 30)), "pv_shift": 35}
    ref = np.stack([oracle.attention(qkv[b], gh, gw, wh, ww, H, 32, p["score_mult"],
                                     p["score_shift"], p["smax_I0"], p["pv_mult"],
                                     p["pv_shift"]) for b in range(B)])
    got = host(ilw.ilw_attention(dev(qkv), gh, gw, wh, ww, H, p))
    assert_same(got, ref, "attention hd32")


# (k_inter, k_out, I0, s_d): rows whose tiny S_sum makes F >= 2^(32 - k_out
# + s_d) (k_inter = 4 with I0 = 1 or 2), output shifts on both sides of 32
# (s_d = 7 and 9 at k_out = 8), and other output widths.
SMAX_PARAMS = [(4, 8, 1, -1), (4, 8, 2, 0), (16, 5, 8, -1), (16, 2, 16, -1), (10, 8, 100, 3),
               (16, 8, 24, 9), (16, 8, 24, 7)]


@pytest.mark.parametrize("case", [(2, 10, 10, 5, 5, 2), (4, 40, 40, 20, 20, 3),
                                  (1, 40, 40, 0, 0, 3)])
@pytest.mark.parametrize("smax", SMAX_PARAMS)
def test_attention_shiftmax_params(case, smax):
    _attention_smax_case(case, smax)


@pytest.mark.parametrize("smax", [SMAX_PARAMS[0], SMAX_PARAMS[5]])
def test_attention_shiftmax_params_large_grid(smax):
    _attention_smax_case((4, 40, 40, 0, 0, 3), smax)


def _attention_smax_case(case, smax):
    B, gh, gw, wh, ww, H = case
    k_inter, k_out, I0, s_d = smax
    say(f"attention smax k_inter={k_inter} k_out={k_out} I0={I0} s_d={s_d} B={B} "
        f"grid={gh}x{gw} win={wh}x{ww} heads={H}")
    g = rng(gh * 7 + wh + I0 + k_out)
    D, T = 64 * H, gh * gw
    qkv = g.integers(-127, 128, (B, T, 3 * D)).astype(np.int8)
    p = {"score_mult": int(g.integers(2 ** 29, 2 ** 30)), "score_shift": 39, "smax_I0": I0,
         "smax_k_inter": k_inter, "smax_k_out": k_out, "smax_s_d": s_d,
         "pv_mult": int(g.integers(2 ** 29, 2 ** 30)), "pv_shift": 30 + k_out}
    ref = np.stack([oracle.attention(qkv[b], gh, gw, wh, ww, H, 64, p["score_mult"],
                                     p["score_shift"], I0, p["pv_mult"], p["pv_shift"],
                                     k_inter=k_inter, k_out=k_out, s_d=s_d)
                    for b in range(B)])
    got = host(ilw.ilw_attention(dev(qkv), gh, gw, wh, ww, H, p))
    assert_same(got, ref, "attention shiftmax params")


@pytest.mark.parametrize("case", [(1, 40, 40, 0, 0, 1), (2, 40, 40, 20, 20, 1),
                                  (1, 6, 10, 3, 5, 1)])
def test_attention_large_m_p(case):
    """m_p = 31 with I0 = 16383: s_d reaches 41 on 1600-token rows, past the
    64-bit range of the output shift."""
    B, gh, gw, wh, ww, H = case
    say(f"attention m_p=31 I0=16383 B={B} grid={gh}x{gw} win={wh}x{ww}")
    g = rng(gh * gw + wh)
    D, T = 64 * H, gh * gw
    qkv = g.integers(-127, 128, (B, T, 3 * D)).astype(np.int8)
    qkv[:, : T // 2, :D] = 0  # rows of equal scores beside random ones
    p = {"score_mult": int(g.integers(2 ** 29, 2 ** 30)), "score_shift": 39,
         "smax_I0": 16383, "smax_m_p": 31, "smax_s_d": -1,
         "pv_mult": int(g.integers(2 ** 29, 2 ** 30)), "pv_shift": 30}
    ref = np.stack([oracle.attention(qkv[b], gh, gw, wh, ww, H, 64, p["score_mult"],
                                     p["score_shift"], 16383, p["pv_mult"], p["pv_shift"],
                                     m_p=31) for b in range(B)])
    got = host(ilw.ilw_attention(dev(qkv), gh, gw, wh, ww, H, p))
    assert_same(got, ref, "attention large m_p")


@pytest.mark.parametrize("case", [(4, 40, 40, 20, 20, 3), (1, 40, 40, 0, 0, 3),
                                  (4, 40, 40, 0, 0, 3)])
@pytest.mark.parametrize("I0", [1023, 1500, 2047])
@pytest.mark.parametrize("zero_q", [False, True])
def test_attention_large_I0(case, I0, zero_q):
    """Large ShiftExp scales (ShiftExp(0) = I0 * 2^16 up to 2^27) on the
    variants whose lanes sum up to 64 values of a row (32-row blocks of
    400-token windows; 1600-token rows on small and large grids): 32-bit
    partial sums are exact only up to I0 = 1023.  Zero queries make every
    score equal, so every value is ShiftExp(0)."""
    B, gh, gw, wh, ww, H = case
    say(f"attention large I0={I0} zero_q={zero_q} B={B} grid={gh}x{gw} win={wh}x{ww}")
    g = rng(I0 + gh * wh + B)
    D, T = 64 * H, gh * gw
    qkv = g.integers(-127, 128, (B, T, 3 * D)).astype(np.int8)
    if zero_q:
        qkv[:, :, :D] = 0
    p = {"score_mult": int(g.integers(2 ** 29, 2 ** 30)), "score_shift": 39,
         "smax_I0": I0, "smax_s_d": -1,
         "pv_mult": int(g.integers(2 ** 29, 2 ** 30)), "pv_shift": 36}
    ref = np.stack([oracle.attention(qkv[b], gh, gw, wh, ww, H, 64, p["score_mult"],
                                     p["score_shift"], I0, p["pv_mult"], p["pv_shift"])
                    for b in range(B)])
    got = host(ilw.ilw_attention(dev(qkv), gh, gw, wh, ww, H, p))
    assert_same(got, ref, "attention large I0")


# ------------------------------------------------------------------ encoder block
@pytest.mark.parametrize("variant", ["wide", "baseline"])
def test_block_c1(variant):
    say(f"block_t256_d192 variant={variant}")
    wl = synth.WORKLOADS["block_t256_d192"]
    blocks, x = synth.encoder_inputs(wl, 101, variant)
    ref = oracle.block_forward(blocks[0], x, 16, 16, 0, 0)
    blk = ilw.DeviceBlock(blocks[0])
    got = host(ilw.ilw_block_forward(blk, dev(x), 16, 16, 0, 0))
    assert_same(got, ref, "block")


@pytest.mark.parametrize("dims,grid,win,B", [((128, 2, 512), (8, 12), (4, 6), 3),
                                              ((192, 3, 768), (10, 10), (5, 5), 2),
                                              ((64, 1, 16), (3, 7), (0, 0), 1)])
def test_block_shapes(dims, grid, win, B):
    D, H, Hm = dims
    say(f"block D={D} H={H} mlp={Hm} grid={grid} win={win} B={B}")
    p = synth.block_params(rng(D + Hm), D, H, 64, Hm, "wide", ln_iters=20, smax_s_d=-1)
    x = rng(7).integers(-127, 128, (B, grid[0] * grid[1], D)).astype(np.int8)
    ref = oracle.block_forward(p, x, *grid, *win)
    blk = ilw.DeviceBlock(p)
    t = dev(x)
    got = host(ilw.ilw_block_forward(blk, t, *grid, *win, y=t))  # in place
    assert_same(got, ref, "block in place")


@pytest.mark.parametrize("dims,B,win", [((384, 6, 1536), 9, (20, 20)), ((384, 6, 1536), 9, (0, 0)),
                                        ((256, 4, 1024), 11, (20, 20))])
def test_block_large_unpacked(dims, B, win):
    """One block through the block entry point (weights not packed) on grids
    past the GEMM latency mode: the throughput QKV, fused-LayerNorm (128-byte
    K steps at 384 channels) and GELU tiles; two images against the oracle."""
    D, H, Hm = dims
    grid = (40, 40)
    say(f"block large D={D} B={B} win={win}")
    p = synth.block_params(rng(D + B), D, H, 64, Hm, "baseline", ln_iters=10, smax_s_d=-1)
    x = rng(8 + B).integers(-127, 128, (B, grid[0] * grid[1], D)).astype(np.int8)
    got = host(ilw.ilw_block_forward(ilw.DeviceBlock(p), dev(x), *grid, *win))
    for b in (0, B - 1):
        ref = oracle.block_forward(p, x[b:b + 1], *grid, *win)
        assert_same(got[b:b + 1], ref, f"block large image {b}")


@pytest.mark.parametrize("dims", [(128, 2, 512), (384, 6, 1536)])
def test_block_requant_fallback(dims):
    """A block whose QKV, projection, fc1 and fc2 layers each hold a channel
    with a large shift (44 to 47) or a bias of 2^21 or more."""
    D, H, Hm = dims
    say(f"block requant fallback D={D}")
    p = synth.block_params(rng(D + 5), D, H, 64, Hm, "wide", ln_iters=20, smax_s_d=-1)
    p["qkv_shift"][7] = 44
    p["proj_shift"][3] = 47
    p["b_fc1"][100] = 1 << 22
    p["fc2_shift"][5] = 45
    p["b_fc2"][9] = -(1 << 21)
    x = rng(8).integers(-127, 128, (2, 96, D)).astype(np.int8)
    ref = oracle.block_forward(p, x, 8, 12, 4, 6)
    got = host(ilw.ilw_block_forward(ilw.DeviceBlock(p), dev(x), 8, 12, 4, 6))
    assert_same(got, ref, "block requant fallback")


# Biases near the int32 limits that still keep b + sum(x w) inside int32
# (the method's int32 accumulator; |sum| <= 1536 * 127^2 < 2^25 here).
BIG_BIAS = [(1 << 31) - (1 << 25), -(1 << 31) + (1 << 25), 1 << 30, -(1 << 30), 1 << 21]


def test_linear_extreme_biases():
    """Biases near the int32 limits, with every shift form (30..43, 44..53,
    62)."""
    say("linear extreme biases")
    g = rng(31)
    M, N, K = 300, 128, 768
    x = g.integers(-127, 128, (M, K)).astype(np.int8)
    w = g.integers(-127, 128, (N, K)).astype(np.int8)
    bias = g.integers(-2 ** 15, 2 ** 15 + 1, N).astype(np.int32)
    mult = g.integers(2 ** 29, 2 ** 30 + 1, N).astype(np.int32)
    shift = g.integers(30, 44, N).astype(np.int32)
    for i in range(0, N, 7):
        bias[i] = BIG_BIAS[(i // 7) % len(BIG_BIAS)]
        shift[i] = (30, 37, 43, 50, 53, 62)[(i // 7) % 6]
        mult[i] = (1 << 31) - 1 if i % 2 else 3
    ref = oracle.linear(x, w, bias, mult, shift)
    got = host(ilw.ilw_linear(dev(x), dev(w), dev(bias), dev(mult), dev(shift)))
    assert_same(got, ref, "linear extreme biases")


@pytest.mark.parametrize("dims", [(192, 3, 768), (384, 6, 1536)])
def test_block_extreme_biases(dims):
    """A block (192 channels: the head and tail kernels; 384: the linears)
    whose QKV, projection, fc1 and fc2 biases include values near +-2^31."""
    D, H, Hm = dims
    say(f"block extreme biases D={D}")
    p = synth.block_params(rng(D + 9), D, H, 64, Hm, "wide", ln_iters=10, smax_s_d=-1)
    for k, n in (("b_qkv", 3 * D), ("b_proj", D), ("b_fc1", Hm), ("b_fc2", D)):
        for j, b in enumerate(BIG_BIAS):
            p[k][(j * 37 + 5) % n] = b
    x = rng(9).integers(-127, 128, (1, 96, D)).astype(np.int8)
    ref = oracle.block_forward(p, x, 8, 12, 4, 6)
    got = host(ilw.ilw_block_forward(ilw.DeviceBlock(p), dev(x), 8, 12, 4, 6))
    assert_same(got, ref, "block extreme biases")


def encoder_ref(blocks, windows, x, gh, gw):
    for p, (wh, ww) in zip(blocks, windows):
        x = oracle.block_forward(p, x, gh, gw, wh, ww)
    return x


@pytest.mark.parametrize("variant", ["wide", "baseline"])
def test_encoder_c2_full(variant):
    """The 6-block tiny encoder at batch 1, every output compared."""
    wl = synth.WORKLOADS["encoder_t1600_d192_b1"]
    say(f"{wl.name} variant={variant}")
    blocks, x = synth.encoder_inputs(wl, 2, variant)
    ref = encoder_ref(blocks, wl.windows, x, wl.grid_h, wl.grid_w)
    enc = ilw.Encoder(blocks, wl.windows, wl.grid_h, wl.grid_w)
    got = host(enc.forward(dev(x)))
    assert_same(got, ref, "encoder c2")


def _oracle_images(blocks, windows, x, gh, gw, images):
    """The oracle encoder of each listed image, on a pool of host threads
    (one image per task: the oracle's C calls release the GIL)."""
    import concurrent.futures as cf
    import os
    threads = max(1, min(16, len(os.sched_getaffinity(0)), len(images)))
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        futs = {b: ex.submit(encoder_ref, blocks, windows, x[b:b + 1], gh, gw) for b in images}
        return {b: f.result() for b, f in futs.items()}


def _encoder_full_batch(name, seed, variant, images=None):
    """The whole batch on the GPU in one call; the listed images (default:
    all) against the oracle, the oracle running while the GPU works."""
    import concurrent.futures as cf
    wl = synth.WORKLOADS[name]
    blocks, x = synth.encoder_inputs(wl, seed, variant)
    images = list(range(wl.batch)) if images is None else images
    say(f"{wl.name} variant={variant}: oracle on {len(images)} images")
    with cf.ThreadPoolExecutor(max_workers=1) as bg:
        refs = bg.submit(_oracle_images, blocks, wl.windows, x, wl.grid_h, wl.grid_w, images)
        enc = ilw.Encoder(blocks, wl.windows, wl.grid_h, wl.grid_w)
        full = host(enc.forward(dev(x)))
        refs = refs.result()
    for b in images:
        assert_same(full[b:b + 1], refs[b], f"{wl.name} {variant} image {b}")
    return wl, blocks, x, full


@pytest.mark.parametrize("name,batch", [("encoder_t1600_d192_b32", 6), ("encoder_t1600_d192_b32", 8),
                                        ("encoder_t1600_d192_b32", 12),
                                        ("encoder_t1600_d384_b8", 3)])
def test_encoder_mid_batches(name, batch):
    """The encoders at batch sizes between the block-tail and throughput
    regimes: the tiny encoder on its separate linears from batch 6 (batch 6
    on the latency-mode LayerNorm tiles, 8 and 12 on the throughput ones, the
    QKV on one-wave 64 x 64 tiles at batch 8), the medium encoder at batch 3
    (the one-kernel block tail on 75 tiles, the QKV on its wide tiles).  The
    first and last images against the oracle."""
    import concurrent.futures as cf
    wl = synth.WORKLOADS[name]
    blocks, x = synth.encoder_inputs(wl, 40 + batch, "baseline", batch=batch)
    images = [0, batch - 1]
    say(f"{wl.name} at batch {batch}: oracle on {len(images)} images")
    with cf.ThreadPoolExecutor(max_workers=1) as bg:
        refs = bg.submit(_oracle_images, blocks, wl.windows, x, wl.grid_h, wl.grid_w, images)
        enc = ilw.Encoder(blocks, wl.windows, wl.grid_h, wl.grid_w)
        full = host(enc.forward(dev(x)))
        refs = refs.result()
    for b in images:
        assert_same(full[b:b + 1], refs[b], f"{wl.name} batch {batch} image {b}")


def test_encoder_c4_full():
    """The tiny encoder at batch 32 (51 200 tokens per layer) with the
    specified parameter distributions: all 32 images against the oracle."""
    _encoder_full_batch("encoder_t1600_d192_b32", 4, "baseline")


def test_encoder_c4_wide_sampled():
    """The same at batch 32 with the wide-shift parameters (rounding paths
    away from saturation): three images against the oracle, every image
    against its own batch-1 GPU run."""
    wl, blocks, x, full = _encoder_full_batch("encoder_t1600_d192_b32", 4, "wide",
                                              images=[0, 17, 31])
    enc = ilw.Encoder(blocks, wl.windows, wl.grid_h, wl.grid_w)
    for b in range(wl.batch):
        one = host(enc.forward(dev(x[b:b + 1])))
        assert_same(full[b:b + 1], one, f"batch independence image {b}")


def test_encoder_c3_full():
    """The 10-block medium encoder at batch 8 with the specified parameter
    distributions (the benchmarked configuration): all 8 images against the
    oracle."""
    _encoder_full_batch("encoder_t1600_d384_b8", 3, "baseline")


def test_encoder_c3_wide_sampled():
    """The medium encoder with the wide-shift parameters: two images against
    the oracle, every image against its own batch-1 GPU run."""
    wl, blocks, x, full = _encoder_full_batch("encoder_t1600_d384_b8", 3, "wide",
                                              images=[2, 5])
    enc = ilw.Encoder(blocks, wl.windows, wl.grid_h, wl.grid_w)
    for b in range(wl.batch):
        one = host(enc.forward(dev(x[b:b + 1])))
        assert_same(full[b:b + 1], one, f"batch independence image {b}")


def _encoder_case(D, H, Hm, depth, seed, variant="wide"):
    g = rng(seed)
    return [synth.block_params(g, D, H, 64, Hm, variant, ln_iters=12 + 4 * (i % 2),
                               smax_s_d=(-1 if i % 2 == 0 else 3)) for i in range(depth)]


@pytest.mark.parametrize("D,H,Hm,grid,windows,B", [
    # 192 and 384 channels: LayerNorm fused into the residual linears
    (192, 3, 768, (9, 12), [(3, 4), (0, 0), (9, 6)], 2),
    (384, 6, 1536, (7, 10), [(0, 0), (7, 5), (0, 0)], 3),
    # 256 channels: fused as well (256-channel LayerNorm tiles)
    (256, 4, 512, (6, 6), [(3, 3), (0, 0)], 2),
    # 128 channels: stand-alone LayerNorm kernels
    (128, 2, 512, (6, 8), [(3, 4), (0, 0)], 2),
    # one block: no next block to fuse LN1 into
    (192, 3, 384, (8, 8), [(4, 4)], 1),
    # 384 channels, 15 tokens: the one-kernel block tail on a single,
    # mostly empty 64-token tile; MLP 768 (two fc1 chunks)
    (384, 6, 768, (3, 5), [(0, 0), (3, 5)], 1),
])
def test_encoder_shapes(D, H, Hm, grid, windows, B):
    """ilw_encoder_forward on ragged token counts against the oracle block
    chain, once into a fresh output and once in place."""
    say(f"encoder D={D} mlp={Hm} grid={grid} windows={windows} B={B}")
    blocks = _encoder_case(D, H, Hm, len(windows), D + Hm + B)
    x = rng(D + 1).integers(-127, 128, (B, grid[0] * grid[1], D)).astype(np.int8)
    ref = encoder_ref(blocks, windows, x, *grid)
    enc = ilw.Encoder(blocks, windows, *grid)
    assert_same(host(enc.forward(dev(x))), ref, "encoder")
    t = dev(x)
    assert_same(host(enc.forward(t, out=t)), ref, "encoder in place")


@pytest.mark.parametrize("D,H", [(192, 3), (384, 6)])
def test_encoder_fused_layernorm_edge_params(D, H):
    """The fused LayerNorms (block tail kernel at D = 192, GEMM epilogue at
    D = 384) with per-tensor output constants, |beta| beyond 2^30 (the 64-bit
    output path), per-tensor linear scales, and one constant input row (zero
    variance)."""
    say(f"encoder fused LN edge parameters D={D}")
    blocks = _encoder_case(D, H, 4 * D, 3, 40 + D)
    g = rng(D)
    blocks[1]["ln1_mult"] = blocks[1]["ln1_mult"][:1].copy()
    blocks[1]["ln1_shift"] = blocks[1]["ln1_shift"][:1].copy()
    for k in ("proj", "fc2", "qkv"):
        blocks[2][k + "_mult"] = blocks[2][k + "_mult"][:1].copy()
        blocks[2][k + "_shift"] = blocks[2][k + "_shift"][:1].copy()
    blocks[1]["ln2_beta"] = g.integers(-2 ** 31 + 1, 2 ** 31 - 1, D).astype(np.int32)
    blocks[2]["ln1_beta"][:4] = [2 ** 31 - 1, -(2 ** 31) + 1, 2 ** 30 + 1, -(2 ** 30) - 1]
    grid, windows = (6, 9), [(3, 3), (0, 0), (2, 3)]
    x = g.integers(-127, 128, (2, 54, D)).astype(np.int8)
    x[1, 7] = 5
    ref = encoder_ref(blocks, windows, x, *grid)
    enc = ilw.Encoder(blocks, windows, *grid)
    assert_same(host(enc.forward(dev(x))), ref, "encoder LN edge parameters")


@pytest.mark.parametrize("shift", [1, 8, 9])
@pytest.mark.parametrize("D,H,B,grid,win", [(192, 3, 1, (16, 16), (8, 8)),
                                            (192, 3, 2, (9, 12), (3, 4)),
                                            (384, 6, 2, (7, 10), (7, 5)),
                                            (128, 2, 2, (6, 8), (3, 4))])
def test_encoder_residual_shift_forms(D, H, B, grid, win, shift):
    """Residual adds with shifts below 9 (the general 64-bit saturation) and
    at 9 (the smallest shift of the 32-bit form), in every residual epilogue:
    the batch-1 block tail (D = 192), the LayerNorm-fused GEMM tiles (192,
    384) and the plain residual tile (128).  Multipliers near 2^shift, except
    one of 2^30 in the second block's first residual, which saturates almost
    every output there."""
    say(f"encoder residual shift {shift} D={D} B={B} grid={grid}")
    windows = [win, (0, 0)]
    blocks = _encoder_case(D, H, 4 * D, 2, 60 + D + shift + B)
    g = rng(70 + shift + D)
    for i, blk in enumerate(blocks):
        blk["res1_shift"] = blk["res2_shift"] = shift
        for k in ("res1_mult_a", "res1_mult_b", "res2_mult_a", "res2_mult_b"):
            blk[k] = int(g.integers(1 << (shift - 1), 3 << (shift - 1)))
        if i == 1:
            blk["res1_mult_a"] = 1 << 30
    x = g.integers(-127, 128, (B, grid[0] * grid[1], D)).astype(np.int8)
    ref = encoder_ref(blocks, windows, x, *grid)
    enc = ilw.Encoder(blocks, windows, *grid)
    assert_same(host(enc.forward(dev(x))), ref, "encoder residual shift forms")


@pytest.mark.parametrize("variant,mlp", [("baseline", 1536), ("wide", 1536), ("baseline", 1024),
                                         ("baseline", 768), ("wide", 1152),
                                         ("wide_big_bias", 1536), ("fc1_clamped", 1536),
                                         ("res_shift_8", 1536), ("res_shift_mixed", 1152),
                                         ("res_shift_8", 1024), ("res_shift_mixed2", 768)])
def test_encoder_384_packed_ragged(variant, mlp):
    """The 384-channel LayerNorm-fused linears on their packed-weight kernel
    (grids past the latency mode: 7 images of 41 x 41 tokens, 11 767 tokens,
    the last 64-token tile 55 rows full): three images of a two-block encoder
    against the oracle, run on host threads while the GPU works.  MLP 1536,
    1152 and 768 run the whole MLP as one kernel (4, 3 and 2 chunks of 384
    fc1 channels; the first block with the next LayerNorm, the second
    without); MLP 1024 runs fc1 and fc2 apart, fc2 with 8 K steps (the
    two-set weight ring).  fc1's requantization skips the accumulator clamp
    unless a channel's shift and |mult| (|bias| + 384 * 2^14) would let the
    shifted value leave int32: 'wide_big_bias' puts biases near +-2^31 on
    that path (shifts 39-42), 'fc1_clamped' adds shifts of 20-23 on some of
    those channels, which sends every tile through the clamp.  Residual
    shifts below 9 take the general 64-bit residual saturation:
    'res_shift_8' in both residual adds (with MLP 1024 on the separate
    LayerNorm-fused linears), 'res_shift_mixed' in the first only (shift 5
    there, 9 in the second), 'res_shift_mixed2' in the second only."""
    import concurrent.futures as cf
    D, H, B, grid, windows = 384, 6, 7, (41, 41), [(0, 0), (0, 0)]
    say(f"encoder D=384 packed weights, {B} images of {grid}, {variant}, MLP {mlp}")
    g = rng(384 + B)
    base = "baseline" if variant == "baseline" else "wide"
    blocks = [synth.block_params(g, D, H, 64, mlp, base, ln_iters=10 + 4 * i,
                                 smax_s_d=(-1 if i == 0 else 5)) for i in range(2)]
    if variant in ("wide_big_bias", "fc1_clamped"):
        for p in blocks:
            for j, b in enumerate(BIG_BIAS):
                n = (j * 131 + 7) % mlp
                p["b_fc1"][n] = b
                if variant == "fc1_clamped":
                    p["fc1_shift"][n] = 20 + j % 4
    if variant.startswith("res_shift"):
        sh1, sh2 = {"res_shift_8": (8, 8), "res_shift_mixed": (5, 9),
                    "res_shift_mixed2": (9, 6)}[variant]
        for p in blocks:
            for r, sh in (("res1", sh1), ("res2", sh2)):
                p[r + "_shift"] = sh
                for k in ("_mult_a", "_mult_b"):
                    p[r + k] = int(g.integers(1 << (sh - 1), 3 << (sh - 1)))
    x = g.integers(-127, 128, (B, grid[0] * grid[1], D)).astype(np.int8)
    images = [0, 3, 6]
    with cf.ThreadPoolExecutor(max_workers=1) as bg:
        refs = bg.submit(_oracle_images, blocks, windows, x, *grid, images)
        enc = ilw.Encoder(blocks, windows, *grid)
        full = host(enc.forward(dev(x)))
        refs = refs.result()
    for b in images:
        assert_same(full[b:b + 1], refs[b], f"encoder 384 packed image {b}")


def test_encoder_big_grid_sampled():
    """A grid large enough for the two-wave-row fused fc2 tile (192 channels,
    deep K), with a ragged token count: sampled images against the oracle."""
    grid, windows = (20, 20), [(10, 10), (0, 0)]
    B = 83  # 33200 tokens: not a multiple of 128
    say(f"encoder big grid B={B}")
    blocks = _encoder_case(192, 3, 768, 2, 77)
    x = rng(78).integers(-127, 128, (B, 400, 192)).astype(np.int8)
    enc = ilw.Encoder(blocks, windows, *grid)
    full = host(enc.forward(dev(x)))
    for b in (0, 41, 82):
        ref = encoder_ref(blocks, windows, x[b:b + 1], *grid)
        assert_same(full[b:b + 1], ref, f"image {b}")


def test_encoder_big_grid_384_sampled():
    """384 channels on a grid large enough for the throughput tiles (the
    128-byte-step LayerNorm tile, the staged QKV and GELU stores), with a
    token count that is a multiple of neither 64 nor 128: sampled images
    against the oracle."""
    grid, windows = (20, 20), [(10, 10), (0, 0)]
    B = 29  # 11600 tokens: more than 1024 waves of 64-token LayerNorm tiles
    say(f"encoder big grid 384 channels B={B}")
    blocks = _encoder_case(384, 6, 1536, 2, 79)
    x = rng(80).integers(-127, 128, (B, 400, 384)).astype(np.int8)
    enc = ilw.Encoder(blocks, windows, *grid)
    full = host(enc.forward(dev(x)))
    for b in (0, 14, 28):
        ref = encoder_ref(blocks, windows, x[b:b + 1], *grid)
        assert_same(full[b:b + 1], ref, f"image {b}")


def test_linear_large_grid_ragged_sampled():
    """A store-epilogue linear on the throughput tiles (output staged through
    LDS) with ragged M and N: the first, last and sampled rows against the
    oracle."""
    M, N, K = 20001, 1040, 192
    say(f"linear large grid M={M} N={N} K={K}")
    g = rng(81)
    x = g.integers(-127, 128, (M, K)).astype(np.int8)
    w = g.integers(-127, 128, (N, K)).astype(np.int8)
    b = g.integers(-2 ** 15, 2 ** 15 + 1, N).astype(np.int32)
    mult = g.integers(2 ** 29, 2 ** 30 + 1, N).astype(np.int32)
    shift = g.integers(36, 44, N).astype(np.int32)
    got = host(ilw.ilw_linear(dev(x), dev(w), dev(b), dev(mult), dev(shift)))
    rows = np.unique(np.concatenate([np.arange(70), np.arange(M - 200, M),
                                     g.integers(0, M, 300)]))
    ref = oracle.linear(x[rows], w, b, mult, shift)
    assert_same(got[rows], ref, "linear large grid rows")


def test_encoder_matches_block_by_block():
    """The encoder entry point (fused LayerNorms) and the block entry point
    give the same bytes."""
    wl = synth.WORKLOADS["encoder_t1600_d192_b1"]
    say("encoder vs block-by-block")
    blocks, x = synth.encoder_inputs(wl, 9, "baseline", batch=3)
    enc = ilw.Encoder(blocks, wl.windows, wl.grid_h, wl.grid_w)
    a = host(enc.forward(dev(x)))
    t = dev(x)
    for blk, w in zip(enc.blocks, wl.windows):
        ilw.ilw_block_forward(blk, t, wl.grid_h, wl.grid_w, *w, y=t)
    assert_same(host(t), a, "encoder vs blocks")


def test_encoder_deterministic():
    wl = synth.WORKLOADS["encoder_t1600_d192_b1"]
    say("encoder determinism")
    blocks, x = synth.encoder_inputs(wl, 8, "baseline", batch=4)
    enc = ilw.Encoder(blocks, wl.windows, wl.grid_h, wl.grid_w)
    a = host(enc.forward(dev(x)))
    b = host(enc.forward(dev(x)))
    assert_same(a, b, "determinism")


# ------------------------------------------------------------------ decoder layer
def _decoder_gpu(p, tgt, mem, ref, hw, start):
    dd = ilw.DeviceDecoder(p)
    return host(ilw.ilw_decoder_layer(dd, dev(tgt), dev(mem), dev(ref), hw, start))


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("shape", [(2, 37, 64, 2, 128, ((9, 13), (4, 6)), 4),
                                   (1, 100, 256, 8, 1024, ((20, 20), (10, 10)), 4),
                                   (3, 16, 128, 2, 256, ((8, 8),), 8)])
def test_decoder_layer_shapes(mode, shape):
    B, Q, D, H, F, levels, P = shape
    say(f"decoder B={B} Q={Q} D={D} H={H} F={F} levels={levels} P={P} mode={mode}")
    wl = synth.DecoderWorkload("t", B, Q, D, H, F, levels, P)
    args = synth.decoder_inputs(wl, Q + D + mode, mode=mode)
    assert_same(_decoder_gpu(*args), oracle.decoder_forward(*args), "decoder")


@pytest.mark.parametrize("mode,B", [(0, 8), (1, 2)])
def test_decoder_layer_c5(mode, B):
    """The decoder layer around the deformable workload: 300 queries, dim 256,
    8 heads of 32, levels 80^2/40^2/20^2, 4 points; every output compared."""
    wl = synth.DECODER_WORKLOADS["decoder_q300_d256_b8"]
    say(f"{wl.name} mode={mode} B={B}")
    args = synth.decoder_inputs(wl, 21 + mode, batch=B, mode=mode)
    assert_same(_decoder_gpu(*args), oracle.decoder_forward(*args), "decoder c5")


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("B,wl_name", [(2, "t"), (8, "decoder_q300_d256_b8")])
def test_decoder_layer_boxes(mode, B, wl_name):
    """The decoder layer with reference boxes (offsets relative to the box),
    at a small shape and at the full 300-query layer."""
    wl = (synth.DECODER_WORKLOADS[wl_name] if wl_name != "t" else
          synth.DecoderWorkload("t", B, 37, 64, 2, 128, ((9, 13), (4, 6)), 4))
    say(f"decoder boxes {wl.name} mode={mode} B={B}")
    args = synth.decoder_inputs(wl, 31 + mode, batch=B, mode=mode, boxes=True)
    assert args[3].shape[-1] == 4
    assert_same(_decoder_gpu(*args), oracle.decoder_forward(*args), "decoder boxes")


# ------------------------------------------------------------------ patch embedding
def _patch_args(d):
    return (d["img"], d["w"], d["bias"], d["mult"], d["shift"], d["pos"], d["pos_mult_a"],
            d["pos_mult_b"], d["pos_shift"])


def _patch_gpu(d):
    return host(ilw.ilw_patch_embed(dev(d["img"]), dev(d["w"]), dev(d["bias"]), dev(d["mult"]),
                                    dev(d["shift"]), dev(d["pos"]), d["pos_mult_a"],
                                    d["pos_mult_b"], d["pos_shift"]))


@pytest.mark.parametrize("B,C,H,W,D", [(1, 3, 640, 640, 192), (2, 3, 48, 32, 32),
                                       (3, 1, 64, 80, 48), (1, 3, 640, 640, 384)])
def test_patch_embed(B, C, H, W, D):
    say(f"patch embed B={B} C={C} {H}x{W} D={D}")
    d = synth.patch_embed_inputs(B + C + D, B, D, H, W, C)
    ref = oracle.patch_embed(*_patch_args(d))
    assert np.std(ref.astype(np.float64)) > 5  # not a constant output
    assert_same(_patch_gpu(d), ref, "patch embed")


def test_patch_embed_b32_sampled():
    """Batch 32 (throughput tiles): three images against the oracle."""
    say("patch embed B=32")
    d = synth.patch_embed_inputs(32, 32, 192)
    got = _patch_gpu(d)
    for b in (0, 15, 31):
        db = dict(d, img=d["img"][b:b + 1])
        assert_same(got[b:b + 1], oracle.patch_embed(*_patch_args(db)), f"image {b}")


def test_patch_embed_offset_output_b16():
    """Throughput tiles (staged residual output) with y only 4 bytes aligned:
    two images against the oracle, guard bytes untouched."""
    say("patch embed B=16, output at a 4-byte offset")
    d = synth.patch_embed_inputs(33, 16, 192)
    T = (d["img"].shape[2] // 16) * (d["img"].shape[3] // 16)
    buf, y = _offset_output((16, T, 192))
    ilw.ilw_patch_embed(dev(d["img"]), dev(d["w"]), dev(d["bias"]), dev(d["mult"]),
                        dev(d["shift"]), dev(d["pos"]), d["pos_mult_a"], d["pos_mult_b"],
                        d["pos_shift"], y=y)
    got = host(y)
    for b in (0, 15):
        db = dict(d, img=d["img"][b:b + 1])
        assert_same(got[b:b + 1], oracle.patch_embed(*_patch_args(db)), f"image {b}")
    rest = host(buf)
    assert np.all(rest[:4] == 0x5a) and np.all(rest[4 + got.size:] == 0x5a), "guard bytes"


def test_encoder_from_image():
    """Image -> patch embedding -> two encoder blocks, against the oracle chain."""
    say("encoder from image")
    d = synth.patch_embed_inputs(9, 2, 192, 160, 160)
    blocks = _encoder_case(192, 3, 768, 2, 10)
    windows = [(5, 5), (0, 0)]
    x0 = oracle.patch_embed(*_patch_args(d))
    ref = encoder_ref(blocks, windows, x0, 10, 10)
    enc = ilw.Encoder(blocks, windows, 10, 10)
    x0d = ilw.ilw_patch_embed(dev(d["img"]), dev(d["w"]), dev(d["bias"]), dev(d["mult"]),
                              dev(d["shift"]), dev(d["pos"]), d["pos_mult_a"], d["pos_mult_b"],
                              d["pos_shift"])
    assert_same(host(enc.forward(x0d)), ref, "encoder from image")


# ------------------------------------------------------------------ I-ViT baselines
@pytest.mark.parametrize("rows,cols", [(1, 1), (7, 4), (300, 400), (64, 1600), (3, 65536)])
@pytest.mark.parametrize("I0,M", [(8, 31), (64, 16), (8192, 31), (24, 32), (16, 8)])
def test_shiftmax_ivit(rows, cols, I0, M):
    say(f"shiftmax ivit rows={rows} cols={cols} I0={I0} M={M}")
    x = rng(rows * 3 + cols + I0).integers(-128, 128, (rows, cols)).astype(np.int8)
    ref = oracle.shiftmax_ivit_rows(x, I0, M=M)
    assert_same(host(ilw.ilw_shiftmax_ivit(dev(x), I0, M=M)), ref, "shiftmax ivit")


def test_shiftmax_ivit_collapse():
    """Rows whose S_sum reaches 2^31 (four equal maxima at I0 = 8192): every
    output 0 on both sides; the constrained kernel keeps the budget."""
    say("shiftmax ivit collapse")
    x = np.zeros((256, 4), np.int8)
    x[::2, 1] = -3
    ref = oracle.shiftmax_ivit_rows(x, 8192, M=31)
    assert np.all(ref[1::2] == 0)
    assert_same(host(ilw.ilw_shiftmax_ivit(dev(x), 8192, M=31)), ref, "collapse")
    got = host(ilw.ilw_shiftmax(dev(x), 8192))
    assert np.all(got[1::2].astype(np.int64).sum(axis=1) >= 120)


@pytest.mark.parametrize("rows,cols", [(1, 1), (333, 768), (64, 1536), (5, 4097)])
@pytest.mark.parametrize("I0", [8, 16, 64])
def test_shiftgelu_ivit(rows, cols, I0):
    say(f"shiftgelu ivit rows={rows} cols={cols} I0={I0}")
    g = rng(rows + cols + I0)
    x = g.integers(-128, 128, (rows, cols)).astype(np.int8)
    x[0] = np.minimum(x[0], 0)  # a row with no positive I_p
    mult, shift = int(g.integers(2 ** 29, 2 ** 30)), int(g.integers(34, 38))
    ref = oracle.shiftgelu_ivit_rows(x, I0, mult, shift)
    assert_same(host(ilw.ilw_shiftgelu_ivit(dev(x), I0, mult, shift)), ref, "shiftgelu ivit")


# ------------------------------------------------------------------ split convolution
def _split_case(g, M, N, chans, per_channel):
    xs = [g.integers(-127, 128, (M, c)).astype(np.int8) for c in chans]
    ws = [g.integers(-127, 128, (N, c)).astype(np.int8) for c in chans]
    nq = N if per_channel else 1
    bm = [g.integers(2 ** 27, 2 ** 30 + 1, nq).astype(np.int32) for _ in chans]
    bs = [np.full(nq, 30, np.int32) for _ in chans]
    bias = g.integers(-2 ** 15, 2 ** 15 + 1, N).astype(np.int32)
    om = g.integers(2 ** 29, 2 ** 30 + 1, nq).astype(np.int32)
    os_ = g.integers(38, 44, nq).astype(np.int32)
    return xs, ws, bm, bs, bias, om, os_


def _split_gpu(xs, ws, bm, bs, bias, om, os_):
    return host(ilw.ilw_split_conv([dev(x) for x in xs], [dev(w) for w in ws],
                                   [dev(m) for m in bm], [dev(v) for v in bs],
                                   None if bias is None else dev(bias), dev(om), dev(os_)))


@pytest.mark.parametrize("M,N,chans", [(1, 16, (64,)), (37, 48, (64, 128)),
                                       (300, 256, (192, 192, 192)),
                                       (1000, 144, (64,) * 8), (129, 32, (384, 64, 192))])
@pytest.mark.parametrize("per_channel", [False, True])
def test_split_conv_shapes(M, N, chans, per_channel):
    say(f"split conv M={M} N={N} chans={chans} per_channel={per_channel}")
    g = rng(M + N + len(chans) + per_channel)
    args = _split_case(g, M, N, chans, per_channel)
    ref = oracle.split_conv(*args)
    assert_same(_split_gpu(*args), ref, "split conv")


def test_split_conv_edge_params():
    """No bias; a branch rescale far above 1 (64-bit running sums, outputs
    saturated through the pre-clamp); a rescale of 1/2 (exact ties)."""
    say("split conv edge parameters")
    g = rng(77)
    xs, ws, bm, bs, _, om, os_ = _split_case(g, 70, 64, (64, 128, 64), True)
    bm[0][:] = 2 ** 31 - 1
    bs[0][:] = 1
    bm[1][:] = 1
    bs[1][:] = 1
    ref = oracle.split_conv(xs, ws, bm, bs, None, om, os_)
    assert np.mean(np.abs(ref) == 127) > 0.5
    assert_same(_split_gpu(xs, ws, bm, bs, None, om, os_), ref, "split conv edge")
    bm[0][:] = 1 << 30
    bs[0][:] = 30
    ref = oracle.split_conv(xs, ws, bm, bs, None, om, os_)
    assert_same(_split_gpu(xs, ws, bm, bs, None, om, os_), ref, "split conv ties")


def _offset_output(shape, off=4):
    """A poisoned device buffer and a view into it at a 4-byte (not 16-byte)
    aligned offset, for outputs that only need 4-byte alignment."""
    n = int(np.prod(shape))
    buf = torch.full((n + 32,), 0x5a, dtype=torch.int8, device="cuda")
    return buf, buf[off:off + n].view(*shape)


def _check_offset_output(buf, got, ref, what, off=4):
    assert_same(got, ref, what)
    rest = host(buf)
    n = ref.size
    assert np.all(rest[:off] == 0x5a) and np.all(rest[off + n:] == 0x5a), f"{what}: guard bytes"


def test_split_conv_offset_output():
    """y only 4 bytes aligned: the staged output takes word stores."""
    say("split conv, output at a 4-byte offset")
    g = rng(83)
    xs, ws, bm, bs, bias, om, os_ = _split_case(g, 300, 128, (64, 128), True)
    ref = oracle.split_conv(xs, ws, bm, bs, bias, om, os_)
    buf, y = _offset_output(ref.shape)
    ilw.ilw_split_conv([dev(a) for a in xs], [dev(a) for a in ws],
                       [dev(a) for a in bm], [dev(a) for a in bs], dev(bias), dev(om),
                       dev(os_), y=y)
    _check_offset_output(buf, host(y), ref, "split conv offset output")


def test_linear_offset_output_large_grid():
    """y only 4 bytes aligned on the throughput tiles (staged output)."""
    M, N, K = 8192, 576, 192
    say(f"linear offset output M={M} N={N} K={K}")
    g = rng(84)
    x = g.integers(-127, 128, (M, K)).astype(np.int8)
    w = g.integers(-127, 128, (N, K)).astype(np.int8)
    b = g.integers(-2 ** 15, 2 ** 15 + 1, N).astype(np.int32)
    mult = g.integers(2 ** 29, 2 ** 30 + 1, N).astype(np.int32)
    shift = g.integers(36, 44, N).astype(np.int32)
    buf, y = _offset_output((M, N))
    ilw.ilw_linear(dev(x), dev(w), dev(b), dev(mult), dev(shift), y=y)
    _check_offset_output(buf, host(y), oracle.linear(x, w, b, mult, shift), "linear offset output")


@pytest.mark.parametrize("per_channel", [False, True])
def test_split_conv_projector_b1_full(per_channel):
    wl = synth.SPLIT_WORKLOADS["splitconv_t1600_c3x192_n256_b1"]
    say(f"{wl.name} per_channel={per_channel}")
    d = synth.split_conv_inputs(wl, 5, per_channel=per_channel)
    args = (d["xs"], d["ws"], d["branch_mults"], d["branch_shifts"], d["bias"],
            d["out_mult"], d["out_shift"])
    assert_same(_split_gpu(*args), oracle.split_conv(*args), "projector b1")


def test_split_conv_projector_b32_sampled():
    """Batch 32 (the large-tile launch): three images against the oracle."""
    wl = synth.SPLIT_WORKLOADS["splitconv_t1600_c3x192_n256_b32"]
    say(wl.name)
    d = synth.split_conv_inputs(wl, 6)
    got = _split_gpu(d["xs"], d["ws"], d["branch_mults"], d["branch_shifts"], d["bias"],
                     d["out_mult"], d["out_shift"])
    T = wl.tokens
    for b in (0, 13, 31):
        rows = slice(b * T, (b + 1) * T)
        ref = oracle.split_conv([x[rows] for x in d["xs"]], d["ws"], d["branch_mults"],
                                d["branch_shifts"], d["bias"], d["out_mult"], d["out_shift"])
        assert_same(got[rows], ref, f"image {b}")


# ------------------------------------------------------------------ deformable sampling
@pytest.mark.parametrize("mode", [0, 1])
def test_deform_c5_full(mode):
    wl = synth.DEFORM_WORKLOADS["deform_q300_d256_b8"]
    say(f"{wl.name} mode={mode}")
    d = synth.deform_inputs(wl, 5)
    ref = oracle.deform_attn(d["value"], d["level_hw"], d["level_start"], d["ref"],
                             d["offsets"], d["logits"], d["I0"], d["out_mult"],
                             d["out_shift"], mode)
    got = host(ilw.ilw_deform_attn(dev(d["value"]), d["level_hw"], d["level_start"],
                                   dev(d["ref"]), dev(d["offsets"]), dev(d["logits"]),
                                   d["I0"], d["out_mult"], d["out_shift"], mode))
    assert_same(got, ref, "deform")
    assert 0 < np.mean(np.abs(ref) == 127) < 0.5


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("s_d", [-1, 2])
def test_deform_shapes(mode, s_d):
    say(f"deform small shapes mode={mode} s_d={s_d}")
    wl = synth.DeformWorkload("small", 3, 7, 48, 3, 16, ((9, 13), (4, 6), (1, 1), (2, 3)), 5)
    d = synth.deform_inputs(wl, 11)
    offs = d["offsets"].copy()
    offs[0, 0] = 0          # exact pixel-grid samples
    offs[1, 2] = 30000      # far outside every level
    ref = oracle.deform_attn(d["value"], d["level_hw"], d["level_start"], d["ref"], offs,
                             d["logits"], 77, 1 << 30, 30, mode, s_d=s_d)
    got = host(ilw.ilw_deform_attn(dev(d["value"]), d["level_hw"], d["level_start"],
                                   dev(d["ref"]), dev(offs), dev(d["logits"]), 77, 1 << 30,
                                   30, mode, s_d=s_d))
    assert_same(got, ref, "deform small")


def _deform_boxes_pair(d, offs, mode, s_d=-1, I0=None, m=None, sh=None):
    I0 = d["I0"] if I0 is None else I0
    m = d["out_mult"] if m is None else m
    sh = d["out_shift"] if sh is None else sh
    ref = oracle.deform_attn(d["value"], d["level_hw"], d["level_start"], d["ref"], offs,
                             d["logits"], I0, m, sh, mode, s_d=s_d)
    got = host(ilw.ilw_deform_attn_boxes(dev(d["value"]), d["level_hw"], d["level_start"],
                                         dev(d["ref"]), dev(offs), dev(d["logits"]), I0, m, sh,
                                         mode, s_d=s_d))
    return got, ref


@pytest.mark.parametrize("mode", [0, 1])
def test_deform_boxes_c5_full(mode):
    """The deformable workload (300 queries, 8 heads, 80^2/40^2/20^2, 4
    points, batch 8) with reference boxes."""
    wl = synth.DEFORM_WORKLOADS["deform_q300_d256_b8"]
    say(f"{wl.name} boxes mode={mode}")
    d = synth.deform_inputs(wl, 55, boxes=True)
    got, ref = _deform_boxes_pair(d, d["offsets"], mode)
    assert_same(got, ref, "deform boxes")
    assert 0 < np.mean(np.abs(ref) == 127) < 0.5


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("P", [5, 4])
def test_deform_boxes_shapes(mode, P):
    """Odd level sizes, P not a power of two, zero offsets, offsets far
    outside, boxes of every size from one pixel to the whole map."""
    say(f"deform boxes small shapes mode={mode} P={P}")
    wl = synth.DeformWorkload("small", 3, 7, 48, 3, 16, ((9, 13), (4, 6), (1, 1), (2, 3)), P)
    d = synth.deform_inputs(wl, 12 + P, boxes=True)
    d["ref"][0, :, 2:] = 1          # tiny boxes
    d["ref"][1, :, 2:] = 65536      # boxes the size of the map
    offs = d["offsets"].copy()
    offs[0, 0] = 0
    offs[2, 3] = 32767
    offs[2, 4] = -32768
    got, ref = _deform_boxes_pair(d, offs, mode, s_d=2 if mode else -1, I0=77, m=1 << 30,
                                  sh=30)
    assert_same(got, ref, "deform boxes small")


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("boxes", [False, True])
@pytest.mark.parametrize("dh,levels,P", [(16, ((9, 13), (4, 6), (2, 3)), 3),   # 4 lanes, 3 samples each
                                          (32, ((9, 13), (4, 6), (2, 3), (1, 1)), 8),  # 8 lanes, 4 each
                                          (64, ((7, 5),), 1),                  # 16 lanes, 1 each
                                          (256, ((6, 6), (3, 3)), 32),         # 64 lanes, 1 each
                                          (8, ((5, 5),), 2),                   # 2 lanes: general kernel
                                          (48, ((5, 4), (2, 2)), 3)])          # 12 lanes: general kernel
def test_deform_lane_groups(mode, boxes, dh, levels, P):
    """Every way the sampler splits a (query, head) over lanes."""
    say(f"deform lane groups dh={dh} levels={levels} P={P} mode={mode} boxes={boxes}")
    heads = 3 if dh < 256 else 1
    wl = synth.DeformWorkload("g", 2, 11, dh * heads, heads, dh, levels, P)
    d = synth.deform_inputs(wl, dh + P, boxes=boxes)
    entry = ilw.ilw_deform_attn_boxes if boxes else ilw.ilw_deform_attn
    ref = oracle.deform_attn(d["value"], d["level_hw"], d["level_start"], d["ref"],
                             d["offsets"], d["logits"], d["I0"], d["out_mult"],
                             d["out_shift"], mode)
    got = host(entry(dev(d["value"]), d["level_hw"], d["level_start"], dev(d["ref"]),
                     dev(d["offsets"]), dev(d["logits"]), d["I0"], d["out_mult"],
                     d["out_shift"], mode))
    assert_same(got, ref, "deform lane groups")


# (k_inter, k_out, m_p, s_d, I0) of the sampling weights' Constrained Shiftmax
DEFORM_SMAX = [(16, 4, 4, -1, 16), (8, 2, 0, -1, 16), (12, 6, 31, -1, 16),
               (16, 8, 4, 20, 16383), (16, 8, 4, 31, 16383), (1, 3, 4, 0, 1),
               (16, 8, 31, -1, 1)]


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("dh,boxes", [(32, False), (32, True), (48, True)])
@pytest.mark.parametrize("smax", DEFORM_SMAX)
def test_deform_shiftmax_params(smax, dh, boxes, mode):
    """Every Constrained Shiftmax parameter of the sampler away from the
    decoder's defaults: k_out down to 2 (weights 0 or 1), m_p = 31 with the
    per-row s_d (the output shift reaches the 64-bit cap), static s_d up to
    31 with I0 at both ends of its range; the wave-group kernel (32 channels
    per head) and the general one (48).  The output shift is the smallest in
    [20, 40) at which the oracle saturates under a fifth of the outputs."""
    k_inter, k_out, m_p, s_d, I0 = smax
    say(f"deform smax k_inter={k_inter} k_out={k_out} m_p={m_p} s_d={s_d} I0={I0} "
        f"dh={dh} boxes={boxes} mode={mode}")
    levels, P = (((9, 13), (4, 6), (2, 3), (1, 1)), 8) if dh == 32 else (((5, 4), (2, 2)), 3)
    wl = synth.DeformWorkload("g", 2, 11, dh * 3, 3, dh, levels, P)
    d = synth.deform_inputs(wl, dh + P + k_inter + k_out, boxes=boxes)
    entry = ilw.ilw_deform_attn_boxes if boxes else ilw.ilw_deform_attn
    kw = dict(k_inter=k_inter, k_out=k_out, m_p=m_p, s_d=s_d)
    for sh in range(20, 40):
        ref = oracle.deform_attn(d["value"], d["level_hw"], d["level_start"], d["ref"],
                                 d["offsets"], d["logits"], I0, 1 << 30, sh, mode, **kw)
        if np.mean(np.abs(ref) == 127) < 0.2:
            break
    got = host(entry(dev(d["value"]), d["level_hw"], d["level_start"], dev(d["ref"]),
                     dev(d["offsets"]), dev(d["logits"]), I0, 1 << 30, sh, mode, **kw))
    assert_same(got, ref, "deform shiftmax params")


@pytest.mark.parametrize("name,parts,B", [("encoder_t1600_d192_b1", 2, 4),
                                          ("encoder_t1600_d192_b1", 2, 3),
                                          ("encoder_t1600_d192_b1", 3, 5),
                                          ("encoder_t1600_d384_b8", 2, 8),
                                          ("encoder_t1600_d384_b8", 2, 5)])
def test_encoder_batch_split_streams(name, parts, B):
    """The batch split over streams (forked from and joined back into the
    capturing stream), captured into a HIP graph: every replay equals the
    one-stream eager forward, uneven splits included; the medium encoder at
    batch 8 in two halves is the benchmark's default."""
    wl = synth.WORKLOADS[name]
    say(f"encoder batch split over {parts} streams, B={B}")
    blocks, x = synth.encoder_inputs(wl, 8, "wide", batch=B)
    enc = ilw.Encoder(blocks, wl.windows, wl.grid_h, wl.grid_w)
    xd = dev(x)
    ref = host(enc.forward(xd)).copy()
    out = torch.empty_like(xd)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        enc.forward_streams(xd, out, parts)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    assert_same(host(out), ref, "eager split")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        enc.forward_streams(xd, out, parts)
    for i in range(3):
        out.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        assert_same(host(out), ref, f"split replay {i}")
        enc.forward(dev(x[::-1].copy()))  # eager work between replays
        torch.cuda.synchronize()


def test_encoder_graph_replay():
    """The benchmark captures the encoder forward into a HIP graph: every
    replay, interleaved with eager work and synchronizations, must reproduce
    the eager result."""
    wl = synth.WORKLOADS["encoder_t1600_d192_b1"]
    say("encoder graph capture and replay")
    blocks, x = synth.encoder_inputs(wl, 6, "wide", batch=2)
    enc = ilw.Encoder(blocks, wl.windows, wl.grid_h, wl.grid_w)
    xd = dev(x)
    out = torch.empty_like(xd)
    ref = host(enc.forward(xd, out)).copy()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        enc.forward(xd, out)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        enc.forward(xd, out)
    for i in range(4):
        out.fill_(0)
        enc.workspace(2).fill_(0)
        g.replay()
        torch.cuda.synchronize()
        assert_same(host(out), ref, f"replay {i}")
        other = enc.forward(dev(x[::-1].copy()))  # eager work between replays
        torch.cuda.synchronize()
        del other
