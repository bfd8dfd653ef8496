"""Seeded synthetic inputs for the integer encoder block and the deformable
sampling layer.

This module only draws integers.  It holds none of the method's arithmetic, so
the tests can feed the same arrays to the CPU oracle and to the GPU library.
Shapes follow the detector the paper quantizes: a ViT encoder on a 640x640
image with patch size 16 (40x40 = 1600 tokens), window and global attention,
and a multi-scale deformable decoder layer.  No dataset is used.

Distributions (all integer-uniform, inclusive):
  int8 activations and weights   [-127, 127]
  int32 GEMM biases              [-2^15, 2^15]
  GEMM dyadic multipliers        [2^29, 2^30]; shifts see ``SHIFTS``
  Shiftmax / GELU I0             [8, 64]
  LayerNorm beta                 [-2^26, 2^26] (scale of the normalized value)
  LayerNorm multipliers          +-[2^29, 2^30] (about 1 in 8 negative: the
                                 multiplier carries gamma, which may be < 0)
  residual multipliers           [2^29, 2^30], shift 31
Draw order: block parameters in struct order, then the block input.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# Shift ranges per requantization point.  "baseline" is the distribution the
# headline workload is specified with (GEMM shifts 30..38, which saturates many
# outputs); "wide" keeps most values inside int8 so that the rounding paths are
# exercised by the parity tests.
SHIFTS = {
    "baseline": {"gemm": (30, 38), "gemm_k4": (30, 38), "score": (30, 38),
                 "pv": (30, 38), "gelu": (35, 38), "ln": (49, 51)},
    "wide": {"gemm": (39, 42), "gemm_k4": (40, 43), "score": (38, 41),
             "pv": (34, 37), "gelu": (34, 37), "ln": (49, 51)},
}


@dataclass(frozen=True)
class EncoderWorkload:
    name: str
    batch: int
    grid_h: int
    grid_w: int
    dim: int
    heads: int
    head_dim: int
    mlp_dim: int
    # per block: (win_h, win_w); (0, 0) is global attention
    windows: tuple = field(default_factory=tuple)

    @property
    def tokens(self) -> int:
        return self.grid_h * self.grid_w

    def gemm_ops(self) -> int:
        """Algorithmic int8 ops (2*M*N*K) of one forward over all blocks: the
        QKV, projection and MLP linears, plus Q K^T and P V per window."""
        T, D, Hm, B = self.tokens, self.dim, self.mlp_dim, self.batch
        linear = 2 * T * D * (3 * D + D + Hm + Hm)
        ops = 0
        for wh, ww in self.windows:
            tw = T if wh == 0 else wh * ww
            n_win = T // tw
            attn = 2 * 2 * n_win * tw * tw * D  # QK^T and PV over all heads
            ops += linear + attn
        return ops * B


@dataclass(frozen=True)
class DeformWorkload:
    name: str
    batch: int
    queries: int
    dim: int
    heads: int
    head_dim: int
    levels: tuple  # ((H, W), ...)
    points: int


@dataclass(frozen=True)
class SplitConvWorkload:
    """Projector input convolution: `branches` encoder feature maps of the
    given channel counts, each with its own activation scale, to `out`
    channels, over batch x tokens positions."""
    name: str
    batch: int
    tokens: int
    branches: tuple  # channels per branch
    out: int

    def gemm_ops(self) -> int:
        return 2 * self.batch * self.tokens * self.out * sum(self.branches)


def _alt(n, win):
    """n blocks alternating window / global, window first."""
    return tuple(win if i % 2 == 0 else (0, 0) for i in range(n))


WORKLOADS = {
    # one integer ViT block, 16x16 tokens, global attention
    "block_t256_d192": EncoderWorkload("block_t256_d192", 1, 16, 16, 192, 3, 64,
                                       768, ((0, 0),)),
    # ViT-tiny-shaped encoder on 640x640 / patch 16, 6 blocks, 2x2 windows of
    # 20x20 tokens alternating with global attention
    "encoder_t1600_d192_b1": EncoderWorkload("encoder_t1600_d192_b1", 1, 40, 40,
                                             192, 3, 64, 768, _alt(6, (20, 20))),
    # medium-shaped encoder, 10 blocks, batch 8
    "encoder_t1600_d384_b8": EncoderWorkload("encoder_t1600_d384_b8", 8, 40, 40,
                                             384, 6, 64, 1536, _alt(10, (20, 20))),
    # the tiny encoder at batch 32 (51200 tokens per layer)
    "encoder_t1600_d192_b32": EncoderWorkload("encoder_t1600_d192_b32", 32, 40, 40,
                                              192, 3, 64, 768, _alt(6, (20, 20))),
}

DEFORM_WORKLOADS = {
    "deform_q300_d256_b8": DeformWorkload("deform_q300_d256_b8", 8, 300, 256, 8, 32,
                                          ((80, 80), (40, 40), (20, 20)), 4),
}

# Stage three: the projector's split convolution over three 192-channel
# feature maps of the tiny encoder (40x40 tokens) to 256 channels
SPLIT_WORKLOADS = {
    "splitconv_t1600_c3x192_n256_b1": SplitConvWorkload("splitconv_t1600_c3x192_n256_b1", 1,
                                                        1600, (192, 192, 192), 256),
    "splitconv_t1600_c3x192_n256_b32": SplitConvWorkload("splitconv_t1600_c3x192_n256_b32", 32,
                                                         1600, (192, 192, 192), 256),
}

# Config order of the five workloads (encoder block, tiny encoder, medium
# encoder, tiny encoder at batch 32, deformable layer).
CONFIG_ORDER = ["block_t256_d192", "encoder_t1600_d192_b1", "encoder_t1600_d384_b8",
                "encoder_t1600_d192_b32", "deform_q300_d256_b8"]


def _u(rng, lo, hi, shape=None, dtype=np.int32):
    return rng.integers(lo, hi, size=shape, endpoint=True).astype(dtype)


def _dy(rng, n, shift_range):
    mult = _u(rng, 1 << 29, 1 << 30, n)
    shift = _u(rng, shift_range[0], shift_range[1], n)
    return mult, shift


def block_params(rng: np.random.Generator, dim: int, heads: int, head_dim: int,
                 mlp_dim: int, variant: str = "baseline", ln_iters: int = 10,
                 smax_s_d: int = -1) -> dict:
    """Parameters of one integer encoder block, drawn in struct order."""
    sh = SHIFTS[variant]
    D, Hm = dim, mlp_dim
    p = {"dim": D, "heads": heads, "head_dim": head_dim, "mlp_dim": Hm,
         "ln_iters": ln_iters}

    def ln(prefix):
        p[prefix + "_beta"] = _u(rng, -(1 << 26), 1 << 26, D)
        mag = _u(rng, 1 << 29, 1 << 30, D)
        sign = np.where(rng.integers(0, 8, size=D) == 0, -1, 1).astype(np.int32)
        p[prefix + "_mult"] = (mag * sign).astype(np.int32)
        p[prefix + "_shift"] = _u(rng, sh["ln"][0], sh["ln"][1], D)

    def lin(prefix, n, k, rng_key):
        p["w_" + prefix] = _u(rng, -127, 127, (n, k), np.int8)
        p["b_" + prefix] = _u(rng, -(1 << 15), 1 << 15, n)
        p[prefix + "_mult"], p[prefix + "_shift"] = _dy(rng, n, sh[rng_key])

    ln("ln1")
    lin("qkv", 3 * D, D, "gemm")
    p["score_mult"], p["score_shift"] = (int(v[0]) for v in _dy(rng, 1, sh["score"]))
    p["smax_I0"] = int(_u(rng, 8, 64))
    p["smax_k_inter"], p["smax_k_out"], p["smax_m_p"] = 16, 8, 4
    p["smax_s_d"] = smax_s_d
    p["pv_mult"], p["pv_shift"] = (int(v[0]) for v in _dy(rng, 1, sh["pv"]))
    lin("proj", D, D, "gemm")
    p["res1_mult_a"] = int(_u(rng, 1 << 29, 1 << 30))
    p["res1_mult_b"] = int(_u(rng, 1 << 29, 1 << 30))
    p["res1_shift"] = 31
    ln("ln2")
    lin("fc1", Hm, D, "gemm")
    p["gelu_I0"] = int(_u(rng, 8, 64))
    p["gelu_k_inter"], p["gelu_k_out"] = 16, 8
    p["gelu_mult"], p["gelu_shift"] = (int(v[0]) for v in _dy(rng, 1, sh["gelu"]))
    lin("fc2", D, Hm, "gemm_k4")
    p["res2_mult_a"] = int(_u(rng, 1 << 29, 1 << 30))
    p["res2_mult_b"] = int(_u(rng, 1 << 29, 1 << 30))
    p["res2_shift"] = 31
    return p


def encoder_inputs(wl: EncoderWorkload, seed: int, variant: str = "baseline",
                   batch: int | None = None):
    """Returns (list of block parameter dicts, int8 input [B, T, D])."""
    rng = np.random.Generator(np.random.PCG64(seed))
    blocks = [block_params(rng, wl.dim, wl.heads, wl.head_dim, wl.mlp_dim, variant)
              for _ in wl.windows]
    B = wl.batch if batch is None else batch
    x = _u(rng, -127, 127, (B, wl.tokens, wl.dim), np.int8)
    return blocks, x


def deform_inputs(wl: DeformWorkload, seed: int, batch: int | None = None,
                  queries: int | None = None, boxes: bool = False) -> dict:
    """Inputs of the deformable sampling core: value maps, Q16 reference
    points, Q8 pixel offsets (+-8 px, so some samples leave the map), logits
    over the L*P samples, and the output requantization.  With boxes, the
    references are boxes (cx, cy, w, h): the same centres, sizes U[2^12, 2^15]
    (1/16 to 1/2 of the map), drawn after everything else; the offsets are
    then in Q8 units of size / (2 P), so +-8 units reach +-size / P."""
    rng = np.random.Generator(np.random.PCG64(seed))
    B = wl.batch if batch is None else batch
    Q = wl.queries if queries is None else queries
    L, P, H, Dh = len(wl.levels), wl.points, wl.heads, wl.head_dim
    level_hw = np.array(wl.levels, np.int32).reshape(L, 2)
    sizes = level_hw[:, 0] * level_hw[:, 1]
    level_start = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(np.int32)
    S = int(sizes.sum())
    d = {
        "level_hw": level_hw,
        "level_start": level_start,
        "value": _u(rng, -127, 127, (B, S, H, Dh), np.int8),
        "ref": _u(rng, 0, 65535, (B, Q, 2)),
        "offsets": _u(rng, -2048, 2048, (B, Q, H, L, P, 2), np.int16),
        "logits": _u(rng, -127, 127, (B, Q, H, L * P), np.int8),
        "I0": 16,
    }
    d["out_mult"] = int(_u(rng, 1 << 29, 1 << 30))
    d["out_shift"] = int(_u(rng, 33, 36))
    if boxes:
        d["ref"] = np.concatenate([d["ref"], _u(rng, 1 << 12, 1 << 15, (B, Q, 2))], axis=-1)
    return d


def int8_tensor(seed: int, shape, lo: int = -127, hi: int = 127) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    return _u(rng, lo, hi, shape, np.int8)


def split_conv_inputs(wl: SplitConvWorkload, seed: int, batch: int | None = None,
                      per_channel: bool = False) -> dict:
    """Inputs of the split convolution: int8 feature maps and weights per
    branch; each branch's activation scale drawn in [0.005, 0.05], its rescale
    dyadic m / 2^30 ~ S_b / max(S) (per-channel variant: a per-channel weight
    scale ratio in [0.5, 1] on top); int32 bias; output dyadic with mult
    U[2^29, 2^30] and shift U[40, 44]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    B = wl.batch if batch is None else batch
    M, N = B * wl.tokens, wl.out
    xs = [_u(rng, -127, 127, (M, c), np.int8) for c in wl.branches]
    ws = [_u(rng, -127, 127, (N, c), np.int8) for c in wl.branches]
    scales = rng.uniform(0.005, 0.05, len(wl.branches))
    top = scales.max()
    bm, bs = [], []
    for sb in scales:
        ratio = sb / top
        if per_channel:
            ratio = ratio * rng.uniform(0.5, 1.0, N)
        m = np.round(np.atleast_1d(ratio) * (1 << 30)).astype(np.int64)
        bm.append(np.minimum(m, (1 << 30)).astype(np.int32))
        bs.append(np.full(m.shape, 30, np.int32))
    bias = _u(rng, -(1 << 15), 1 << 15, N)
    om = _u(rng, 1 << 29, 1 << 30, N)
    os_ = _u(rng, 40, 44, N)
    return {"xs": xs, "ws": ws, "branch_mults": bm, "branch_shifts": bs, "bias": bias,
            "out_mult": om, "out_shift": os_, "scales": scales}


def patch_embed_inputs(seed: int, batch: int, dim: int, height: int = 640, width: int = 640,
                       channels: int = 3, shift_range=(40, 43)) -> dict:
    """Patch-embedding inputs: an int8 image U[-127, 127] (a per-tensor
    quantized RGB frame), 16x16 patch weights [dim, channels*256] with int32
    bias and per-channel dyadic (mult U[2^29, 2^30], shift in shift_range),
    an int8 positional table [T, dim] and its add (mults U[2^29, 2^30],
    shift 31)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    T = (height // 16) * (width // 16)
    return {
        "img": _u(rng, -127, 127, (batch, channels, height, width), np.int8),
        "w": _u(rng, -127, 127, (dim, channels * 256), np.int8),
        "bias": _u(rng, -(1 << 15), 1 << 15, dim),
        "mult": _u(rng, 1 << 29, 1 << 30, dim),
        "shift": _u(rng, shift_range[0], shift_range[1], dim),
        "pos": _u(rng, -127, 127, (T, dim), np.int8),
        "pos_mult_a": int(_u(rng, 1 << 29, 1 << 30)),
        "pos_mult_b": int(_u(rng, 1 << 29, 1 << 30)),
        "pos_shift": 31,
    }


@dataclass(frozen=True)
class DecoderWorkload:
    """One integer deformable decoder layer: queries of dim `dim` over the
    stacked encoder maps of `levels`."""
    name: str
    batch: int
    queries: int
    dim: int
    heads: int
    ffn_dim: int
    levels: tuple
    points: int

    def gemm_ops(self) -> int:
        B, Q, D, H, F = self.batch, self.queries, self.dim, self.heads, self.ffn_dim
        L, P = len(self.levels), self.points
        S = sum(h * w for h, w in self.levels)
        lin = 2 * B * Q * D * (3 * D + D + H * L * P * 3 + D + 2 * F) + 2 * B * S * D * D
        attn = 4 * B * Q * Q * D
        return lin + attn


DECODER_WORKLOADS = {
    "decoder_q300_d256_b8": DecoderWorkload("decoder_q300_d256_b8", 8, 300, 256, 8, 1024,
                                            ((80, 80), (40, 40), (20, 20)), 4),
}


def decoder_params(rng: np.random.Generator, dim: int, heads: int, ffn_dim: int,
                   levels: int, points: int, ln_iters: int = 20, mode: int = 0) -> dict:
    """Parameters of one integer decoder layer, drawn in struct order (the
    'wide' GEMM shifts so that most values stay inside int8; the offset
    linear's shift spreads offsets over the int8 range, i.e. +-8 px at
    1/16 px)."""
    D, H, F, L, P = dim, heads, ffn_dim, levels, points
    sh = SHIFTS["wide"]
    p = {"dim": D, "heads": H, "ffn_dim": F, "levels": L, "points": P, "ln_iters": ln_iters}

    def lin(stem, n, k, key="gemm"):
        p["w_" + stem] = _u(rng, -127, 127, (n, k), np.int8)
        p["b_" + stem] = _u(rng, -(1 << 15), 1 << 15, n)
        p[stem + "_mult"], p[stem + "_shift"] = _dy(rng, n, sh[key])

    def ln(stem):
        p[stem + "_beta"] = _u(rng, -(1 << 26), 1 << 26, D)
        mag = _u(rng, 1 << 29, 1 << 30, D)
        sign = np.where(rng.integers(0, 8, size=D) == 0, -1, 1).astype(np.int32)
        p[stem + "_mult"] = (mag * sign).astype(np.int32)
        p[stem + "_shift"] = _u(rng, sh["ln"][0], sh["ln"][1], D)

    def res(i):
        p[f"res{i}_mult_a"] = int(_u(rng, 1 << 29, 1 << 30))
        p[f"res{i}_mult_b"] = int(_u(rng, 1 << 29, 1 << 30))
        p[f"res{i}_shift"] = 31

    lin("qkv", 3 * D, D)
    p["score_mult"], p["score_shift"] = (int(v[0]) for v in _dy(rng, 1, sh["score"]))
    p["smax_I0"] = int(_u(rng, 8, 64))
    p["smax_k_inter"], p["smax_k_out"], p["smax_m_p"], p["smax_s_d"] = 16, 8, 4, -1
    p["pv_mult"], p["pv_shift"] = (int(v[0]) for v in _dy(rng, 1, sh["pv"]))
    lin("o", D, D)
    res(1)
    ln("ln1")
    lin("val", D, D)
    lin("off", H * L * P * 2, D)
    lin("attw", H * L * P, D)
    p["da_I0"], p["da_s_d"] = 16, -1
    p["da_out_mult"] = int(_u(rng, 1 << 29, 1 << 30))
    p["da_out_shift"] = int(_u(rng, 33, 36))  # mode 1 adds the 16 bits of its weights itself
    p["da_mode"] = mode
    lin("co", D, D)
    res(2)
    ln("ln2")
    lin("fc1", F, D)
    p["gelu_I0"], p["gelu_k_inter"], p["gelu_k_out"] = int(_u(rng, 8, 64)), 16, 8
    p["gelu_mult"], p["gelu_shift"] = (int(v[0]) for v in _dy(rng, 1, sh["gelu"]))
    lin("fc2", D, F, "gemm_k4")
    res(3)
    ln("ln3")
    return p


def decoder_inputs(wl: DecoderWorkload, seed: int, batch: int | None = None, mode: int = 0,
                   boxes: bool = False):
    """(params, tgt int8 [B, Q, D], memory int8 [B, S, D], ref int32 Q16
    [B, Q, 2], level_hw [L, 2], level_start [L]).  With boxes, ref is
    [B, Q, 4] (cx, cy, w, h): the same centres, sizes U[2^12, 2^15] drawn
    last."""
    rng = np.random.Generator(np.random.PCG64(seed))
    B = wl.batch if batch is None else batch
    p = decoder_params(rng, wl.dim, wl.heads, wl.ffn_dim, len(wl.levels), wl.points, mode=mode)
    hw = np.array(wl.levels, np.int32)
    start = np.concatenate([[0], np.cumsum(hw[:, 0] * hw[:, 1])[:-1]]).astype(np.int32)
    S = int((hw[:, 0] * hw[:, 1]).sum())
    tgt = _u(rng, -127, 127, (B, wl.queries, wl.dim), np.int8)
    memory = _u(rng, -127, 127, (B, S, wl.dim), np.int8)
    ref = _u(rng, 0, 65535, (B, wl.queries, 2))
    if boxes:
        ref = np.concatenate([ref, _u(rng, 1 << 12, 1 << 15, (B, wl.queries, 2))], axis=-1)
    p["ref_dims"] = ref.shape[-1]
    return p, tgt, memory, ref, hw, start


@dataclass(frozen=True)
class RowOpWorkload:
    """One stand-alone row-wise or element-wise operator over the tensor it
    sees inside the encoder: `rows` x `cols` int8 values."""
    name: str
    op: str  # "shiftmax", "sdshiftgelu", "layernorm", "residual"
    rows: int
    cols: int

    def bytes_moved(self) -> int:
        """Algorithmic HBM bytes of one call: each int8 input read once and
        each output written once (the residual add reads two inputs), plus
        LayerNorm's per-channel beta, multiplier and shift (int32 each)."""
        n = self.rows * self.cols
        if self.op == "residual":
            return 3 * n
        if self.op == "layernorm":
            return 2 * n + 12 * self.cols
        return 2 * n


ROWOP_WORKLOADS = {
    # the score rows of one global attention layer of the tiny encoder at
    # batch 32: 32 images x 3 heads x 1600 queries, rows of 1600 keys
    "shiftmax_r153600_c1600": RowOpWorkload("shiftmax_r153600_c1600", "shiftmax", 153600, 1600),
    # the fc1 output of the tiny encoder at batch 32 (51 200 tokens x 768)
    "sdshiftgelu_r51200_c768": RowOpWorkload("sdshiftgelu_r51200_c768", "sdshiftgelu", 51200,
                                             768),
    # the LayerNorm rows of the medium encoder at batch 8 and of the tiny
    # encoder at batch 32
    "layernorm_r12800_c384": RowOpWorkload("layernorm_r12800_c384", "layernorm", 12800, 384),
    "layernorm_r51200_c192": RowOpWorkload("layernorm_r51200_c192", "layernorm", 51200, 192),
    # the residual add of the tiny encoder at batch 32
    "residual_r51200_c192": RowOpWorkload("residual_r51200_c192", "residual", 51200, 192),
}


def rowop_inputs(wl: RowOpWorkload, seed: int) -> dict:
    """int8 inputs U[-127, 127] and the operator's parameters, drawn as for
    the encoder blocks: Shiftmax and GELU I0 U[8, 64] (k_inter 16, k_out 8,
    m_p 4, dynamic s_d); GELU output dyadic mult U[2^29, 2^30], shift
    U[35, 38]; LayerNorm beta U[-2^26, 2^26], per-channel mult +-U[2^29, 2^30]
    (1 in 8 negative), shift U[49, 51], 10 Newton steps; residual mults
    U[2^29, 2^30], shift 31."""
    rng = np.random.Generator(np.random.PCG64(seed))
    d = {"x": _u(rng, -127, 127, (wl.rows, wl.cols), np.int8)}
    if wl.op == "shiftmax":
        d["I0"] = int(_u(rng, 8, 64))
    elif wl.op == "sdshiftgelu":
        d["I0"] = int(_u(rng, 8, 64))
        d["mult"], d["shift"] = int(_u(rng, 1 << 29, 1 << 30)), int(_u(rng, 35, 38))
    elif wl.op == "layernorm":
        C = wl.cols
        d["beta"] = _u(rng, -(1 << 26), 1 << 26, C)
        mag = _u(rng, 1 << 29, 1 << 30, C)
        sign = np.where(rng.integers(0, 8, size=C) == 0, -1, 1).astype(np.int32)
        d["mult"] = (mag * sign).astype(np.int32)
        d["shift"] = _u(rng, 49, 51, C)
    else:
        d["b"] = _u(rng, -127, 127, (wl.rows, wl.cols), np.int8)
        d["mult_a"], d["mult_b"] = int(_u(rng, 1 << 29, 1 << 30)), int(_u(rng, 1 << 29, 1 << 30))
        d["shift"] = 31
    return d
