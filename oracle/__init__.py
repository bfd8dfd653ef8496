"""CPU oracle for the integer-only I-LW-DETR operators -- TEST INFRASTRUCTURE.

This package loads the plain C oracle (``ilw_oracle.c``) through ctypes.  It is
the slow, obviously-correct reference that the GPU library is checked against.
Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import it; the product package never does, and the oracle
shares no code with it.  Every function is named after the paper's operator and
documented (with the section, equation or algorithm it follows) in the C
source.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ilw_oracle.c")
# ILW_ORACLE_LIBRARY names another build of the same source (the sanitizer
# run of the test-suite loads an instrumented one).
_SO = os.environ.get("ILW_ORACLE_LIBRARY") or os.path.join(_HERE, "libilw_oracle.so")
_LIB = None

i8p = ctypes.POINTER(ctypes.c_int8)
i16p = ctypes.POINTER(ctypes.c_int16)
i32p = ctypes.POINTER(ctypes.c_int32)
i64p = ctypes.POINTER(ctypes.c_int64)
vpp = ctypes.POINTER(ctypes.c_void_p)
c_i32 = ctypes.c_int32
c_i64 = ctypes.c_int64


def build(force: bool = True) -> str:
    """Compile the oracle with plain gcc -O2 (no vectorisation tuning)."""
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared",
                               "-Wall", "-Wextra", "-o", tmp, _SRC])
        os.replace(tmp, _SO)
    return _SO


def build_sanitized(out: str, cc: str) -> str:
    """Compile the oracle with AddressSanitizer and UndefinedBehaviorSanitizer
    (clang, shared sanitizer runtime, abort on the first report) into `out`."""
    subprocess.check_call([cc, "-O1", "-g", "-std=c11", "-fPIC", "-shared",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-fno-omit-frame-pointer", "-shared-libsan", "-o", out, _SRC])
    return out


class OrcBlock(ctypes.Structure):
    """Mirror of the oracle's own ``orc_block`` struct (ilw_oracle.h)."""
    _fields_ = [
        ("dim", c_i32), ("heads", c_i32), ("head_dim", c_i32),
        ("mlp_dim", c_i32), ("ln_iters", c_i32),
        ("ln1_beta", i32p), ("ln1_mult", i32p), ("ln1_shift", i32p),
        ("ln1_nq", c_i32),
        ("w_qkv", i8p), ("b_qkv", i32p), ("qkv_mult", i32p),
        ("qkv_shift", i32p), ("qkv_nq", c_i32),
        ("score_mult", c_i32), ("score_shift", c_i32),
        ("smax_I0", c_i32), ("smax_k_inter", c_i32), ("smax_k_out", c_i32),
        ("smax_m_p", c_i32), ("smax_s_d", c_i32),
        ("pv_mult", c_i32), ("pv_shift", c_i32),
        ("w_proj", i8p), ("b_proj", i32p), ("proj_mult", i32p),
        ("proj_shift", i32p), ("proj_nq", c_i32),
        ("res1_mult_a", c_i32), ("res1_mult_b", c_i32), ("res1_shift", c_i32),
        ("ln2_beta", i32p), ("ln2_mult", i32p), ("ln2_shift", i32p),
        ("ln2_nq", c_i32),
        ("w_fc1", i8p), ("b_fc1", i32p), ("fc1_mult", i32p),
        ("fc1_shift", i32p), ("fc1_nq", c_i32),
        ("gelu_I0", c_i32), ("gelu_k_inter", c_i32), ("gelu_k_out", c_i32),
        ("gelu_mult", c_i32), ("gelu_shift", c_i32),
        ("w_fc2", i8p), ("b_fc2", i32p), ("fc2_mult", i32p),
        ("fc2_shift", i32p), ("fc2_nq", c_i32),
        ("res2_mult_a", c_i32), ("res2_mult_b", c_i32), ("res2_shift", c_i32),
    ]


def _linear_fields(stem):
    return [("w_" + stem, i8p), ("b_" + stem, i32p), (stem + "_mult", i32p),
            (stem + "_shift", i32p), (stem + "_nq", c_i32)]


def _ln_fields(stem):
    return [(stem + "_beta", i32p), (stem + "_mult", i32p), (stem + "_shift", i32p),
            (stem + "_nq", c_i32)]


class OrcDecoder(ctypes.Structure):
    """Mirror of the oracle's own ``orc_decoder`` struct (ilw_oracle.h)."""
    _fields_ = (
        [(n, c_i32) for n in ("dim", "heads", "ffn_dim", "levels", "points", "ln_iters")]
        + _linear_fields("qkv")
        + [(n, c_i32) for n in ("score_mult", "score_shift", "smax_I0", "smax_k_inter",
                                "smax_k_out", "smax_m_p", "smax_s_d", "pv_mult", "pv_shift")]
        + _linear_fields("o")
        + [(n, c_i32) for n in ("res1_mult_a", "res1_mult_b", "res1_shift")]
        + _ln_fields("ln1")
        + _linear_fields("val") + _linear_fields("off") + _linear_fields("attw")
        + [(n, c_i32) for n in ("da_I0", "da_s_d", "da_out_mult", "da_out_shift", "da_mode",
                                "ref_dims")]
        + _linear_fields("co")
        + [(n, c_i32) for n in ("res2_mult_a", "res2_mult_b", "res2_shift")]
        + _ln_fields("ln2")
        + _linear_fields("fc1")
        + [(n, c_i32) for n in ("gelu_I0", "gelu_k_inter", "gelu_k_out", "gelu_mult",
                                "gelu_shift")]
        + _linear_fields("fc2")
        + [(n, c_i32) for n in ("res3_mult_a", "res3_mult_b", "res3_shift")]
        + _ln_fields("ln3"))


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        sig = {
            "orc_floor_div_pow2": (c_i64, [c_i64, c_i32]),
            "orc_requant": (c_i32, [c_i64, c_i32, c_i32]),
            "orc_residual": (c_i32, [c_i32, c_i32, c_i32, c_i32, c_i32]),
            "orc_shiftexp": (c_i64, [c_i64, c_i32, c_i32]),
            "orc_calibrate_shift": (c_i32, [c_i64, c_i32, c_i32]),
            "orc_intdiv": (c_i64, [c_i64, c_i64, c_i32]),
            "orc_sdshiftgelu": (c_i64, [c_i32, c_i32, c_i32, c_i32]),
            "orc_ivit_shiftgelu": (c_i64, [c_i32, c_i32, c_i32, c_i32, c_i32]),
            "orc_isqrt_newton": (c_i64, [c_i64, c_i32]),
            "orc_shiftmax_row": (None, [i32p, c_i32, c_i32, c_i32, c_i32, c_i32,
                                        c_i32, i32p, i64p]),
            "orc_shiftmax_ivit_row": (None, [i32p, c_i32, c_i32, c_i32, c_i32,
                                             c_i32, i32p]),
            "orc_shiftmax_rows": (None, [i8p, i8p, c_i64, c_i32, c_i32, c_i32,
                                         c_i32, c_i32, c_i32]),
            "orc_shiftmax_ivit_rows": (None, [i8p, i8p, c_i64, c_i32, c_i32, c_i32,
                                              c_i32, c_i32]),
            "orc_shiftgelu_ivit_rows": (None, [i8p, i8p, c_i64, c_i32, c_i32, c_i32,
                                               c_i32, c_i32, c_i32]),
            "orc_sdshiftgelu_tensor": (None, [i8p, i8p, c_i64, c_i32, c_i32,
                                              c_i32, c_i32, c_i32]),
            "orc_int_layernorm_row": (None, [i8p, c_i32, i32p, i32p, i32p, c_i32,
                                             c_i32, i8p, i64p]),
            "orc_int_layernorm": (None, [i8p, i8p, c_i64, c_i32, i32p, i32p, i32p,
                                         c_i32, c_i32]),
            "orc_linear_acc": (None, [i8p, i8p, i32p, c_i64, c_i32, c_i32, i32p]),
            "orc_linear": (None, [i8p, i8p, i32p, c_i64, c_i32, c_i32, i32p, i32p,
                                  c_i32, i8p]),
            "orc_residual_tensor": (None, [i8p, i8p, i8p, c_i64, c_i32, c_i32,
                                           c_i32]),
            "orc_split_conv_sum": (None, [c_i32, vpp, i32p, vpp, vpp, vpp, i32p, i32p,
                                          c_i64, c_i32, i64p]),
            "orc_split_conv": (None, [c_i32, vpp, i32p, vpp, vpp, vpp, i32p, i32p, c_i64,
                                      c_i32, i32p, i32p, c_i32, i8p]),
            "orc_patch_embed": (None, [i8p, c_i32, c_i32, c_i32, c_i32, c_i32, i8p, i32p,
                                       i32p, i32p, c_i32, i8p, c_i32, c_i32, c_i32, c_i32,
                                       i8p]),
            "orc_decoder_forward": (None, [ctypes.POINTER(OrcDecoder), i8p, i8p, i32p,
                                           i32p, i32p, c_i32, c_i32, c_i32, i8p]),
            "orc_attention": (None, [i8p] + [c_i32] * 16 + [i8p]),
            "orc_block_forward": (None, [ctypes.POINTER(OrcBlock), i8p, i8p,
                                         c_i32, c_i32, c_i32, c_i32, c_i32]),
            "orc_deform_nearest_index": (c_i64, [c_i32] * 6),
            "orc_deform_box_nearest_index": (c_i64, [c_i32] * 9),
            "orc_deform_attn": (None, [i8p, i32p, i32p, c_i32, c_i32, i32p, i16p,
                                       i8p, i8p] + [c_i32] * 14),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = L
    return _LIB


def _p(a: np.ndarray, t):
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data_as(t)


def _arr(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


# ---------------------------------------------------------------- scalars
def floor_div_pow2(v, s):
    return lib().orc_floor_div_pow2(int(v), int(s))


def requant(acc, mult, shift):
    return lib().orc_requant(int(acc), int(mult), int(shift))


def residual(a, b, mult_a, mult_b, shift):
    return lib().orc_residual(int(a), int(b), int(mult_a), int(mult_b), int(shift))


def shiftexp(I, I0, k_inter=16):
    return lib().orc_shiftexp(int(I), int(I0), int(k_inter))


def calibrate_shift(s_sum, m_p=4, M_hw=31):
    return lib().orc_calibrate_shift(int(s_sum), int(m_p), int(M_hw))


def intdiv(a, b, k_out=8):
    return lib().orc_intdiv(int(a), int(b), int(k_out))


def sdshiftgelu(x, I0, k_inter=16, k_out=8):
    return lib().orc_sdshiftgelu(int(x), int(I0), int(k_inter), int(k_out))


def ivit_shiftgelu(x, max_ip, I0, k_inter=16, k_out=8):
    return lib().orc_ivit_shiftgelu(int(x), int(max_ip), int(I0), int(k_inter),
                                    int(k_out))


def isqrt_newton(V, iters):
    return lib().orc_isqrt_newton(int(V), int(iters))


# ---------------------------------------------------------------- rows / tensors
def shiftmax_row(x, I0, k_inter=16, k_out=8, m_p=4, s_d=-1):
    """Returns (out int32[d], (S_sum, s_d, S_R, F))."""
    x = _arr(x, np.int32)
    out = np.zeros(x.shape[0], np.int32)
    diag = np.zeros(4, np.int64)
    lib().orc_shiftmax_row(_p(x, i32p), x.shape[0], I0, k_inter, k_out, m_p, s_d,
                           _p(out, i32p), _p(diag, i64p))
    return out, tuple(int(v) for v in diag)


def shiftmax_ivit_row(x, I0, k_inter=16, k_out=8, M=31):
    x = _arr(x, np.int32)
    out = np.zeros(x.shape[0], np.int32)
    lib().orc_shiftmax_ivit_row(_p(x, i32p), x.shape[0], I0, k_inter, k_out, M,
                                _p(out, i32p))
    return out


def shiftmax_rows(x, I0, k_inter=16, k_out=8, m_p=4, s_d=-1):
    x = _arr(x, np.int8)
    rows, cols = x.shape
    y = np.zeros_like(x)
    lib().orc_shiftmax_rows(_p(x, i8p), _p(y, i8p), rows, cols, I0, k_inter, k_out,
                            m_p, s_d)
    return y


def sdshiftgelu_tensor(x, I0, out_mult, out_shift, k_inter=16, k_out=8):
    x = _arr(x, np.int8)
    y = np.zeros_like(x)
    lib().orc_sdshiftgelu_tensor(_p(x, i8p), _p(y, i8p), x.size, I0, k_inter, k_out,
                                 out_mult, out_shift)
    return y


def int_layernorm_row(x, beta, mult, shift, iters=10):
    x = _arr(x, np.int8)
    beta, mult, shift = (_arr(a, np.int32) for a in (beta, mult, shift))
    y = np.zeros_like(x)
    diag = np.zeros(4, np.int64)
    lib().orc_int_layernorm_row(_p(x, i8p), x.shape[0], _p(beta, i32p),
                                _p(mult, i32p), _p(shift, i32p), mult.shape[0],
                                iters, _p(y, i8p), _p(diag, i64p))
    return y, tuple(int(v) for v in diag)


def int_layernorm(x, beta, mult, shift, iters=10):
    x = _arr(x, np.int8)
    beta, mult, shift = (_arr(a, np.int32) for a in (beta, mult, shift))
    C = x.shape[-1]
    y = np.zeros_like(x)
    lib().orc_int_layernorm(_p(x, i8p), _p(y, i8p), x.size // C, C, _p(beta, i32p),
                            _p(mult, i32p), _p(shift, i32p), mult.shape[0], iters)
    return y


def linear_acc(x, w, b=None):
    x = _arr(x, np.int8)
    w = _arr(w, np.int8)
    M, K = x.shape
    N = w.shape[0]
    acc = np.zeros((M, N), np.int32)
    bb = _arr(b, np.int32) if b is not None else None
    lib().orc_linear_acc(_p(x, i8p), _p(w, i8p),
                         _p(bb, i32p) if bb is not None else None, M, N, K,
                         _p(acc, i32p))
    return acc


def linear(x, w, b, mult, shift):
    x = _arr(x, np.int8)
    w = _arr(w, np.int8)
    b, mult, shift = (_arr(a, np.int32) for a in (b, mult, shift))
    M, K = x.shape
    N = w.shape[0]
    y = np.zeros((M, N), np.int8)
    lib().orc_linear(_p(x, i8p), _p(w, i8p), _p(b, i32p), M, N, K, _p(mult, i32p),
                     _p(shift, i32p), mult.shape[0], _p(y, i8p))
    return y


def _split_args(xs, ws, br_mults, br_shifts):
    xs = [_arr(x, np.int8) for x in xs]
    ws = [_arr(w, np.int8) for w in ws]
    ms = [_arr(m, np.int32).reshape(-1) for m in br_mults]
    ss = [_arr(v, np.int32).reshape(-1) for v in br_shifts]
    nb = len(xs)
    assert len(ws) == len(ms) == len(ss) == nb >= 1
    M = xs[0].shape[0]
    N = ws[0].shape[0]
    for x, w, m, v in zip(xs, ws, ms, ss):
        assert x.shape[0] == M and w.shape == (N, x.shape[1]) and m.shape == v.shape
        assert m.shape[0] in (1, N)
    ptrs = lambda arrs: (ctypes.c_void_p * nb)(*[a.ctypes.data for a in arrs])
    ch = np.array([x.shape[1] for x in xs], np.int32)
    nq = np.array([m.shape[0] for m in ms], np.int32)
    keep = (xs, ws, ms, ss, ch, nq)
    return keep, nb, M, N, ptrs(xs), ch, ptrs(ws), ptrs(ms), ptrs(ss), nq


def split_conv_sum(xs, ws, br_mults, br_shifts, bias):
    """A = bias + sum_b rescale_b(x_b W_b^T), int64 [M, N] (before the output
    requantization)."""
    keep, nb, M, N, px, ch, pw, pm, ps, nq = _split_args(xs, ws, br_mults, br_shifts)
    b = None if bias is None else _arr(bias, np.int32)
    A = np.zeros((M, N), np.int64)
    lib().orc_split_conv_sum(nb, px, _p(ch, i32p), pw, pm, ps, _p(nq, i32p),
                             None if b is None else _p(b, i32p), M, N, _p(A, i64p))
    return A


def split_conv(xs, ws, br_mults, br_shifts, bias, out_mult, out_shift):
    """Scale-preserving split convolution (pointwise) -> int8 [M, N]."""
    keep, nb, M, N, px, ch, pw, pm, ps, nq = _split_args(xs, ws, br_mults, br_shifts)
    b = None if bias is None else _arr(bias, np.int32)
    om = _arr(out_mult, np.int32).reshape(-1)
    os_ = _arr(out_shift, np.int32).reshape(-1)
    y = np.zeros((M, N), np.int8)
    lib().orc_split_conv(nb, px, _p(ch, i32p), pw, pm, ps, _p(nq, i32p),
                         None if b is None else _p(b, i32p), M, N, _p(om, i32p),
                         _p(os_, i32p), om.shape[0], _p(y, i8p))
    return y


def shiftmax_ivit_rows(x, I0, M=31, k_inter=16, k_out=8):
    """I-ViT Shiftmax (fixed division precision M) of every row of int8 x."""
    x = _arr(x, np.int8)
    rows, cols = x.reshape(-1, x.shape[-1]).shape
    y = np.zeros_like(x)
    lib().orc_shiftmax_ivit_rows(_p(x, i8p), _p(y, i8p), rows, cols, I0, k_inter, k_out, M)
    return y


def shiftgelu_ivit_rows(x, I0, out_mult, out_shift, k_inter=16, k_out=8):
    """I-ViT ShiftGELU (row-maximum shift) of every row of int8 x, requantized."""
    x = _arr(x, np.int8)
    rows, cols = x.reshape(-1, x.shape[-1]).shape
    y = np.zeros_like(x)
    lib().orc_shiftgelu_ivit_rows(_p(x, i8p), _p(y, i8p), rows, cols, I0, k_inter, k_out,
                                  out_mult, out_shift)
    return y


def patch_embed(img, w, bias, mult, shift, pos, pos_ma, pos_mb, pos_shift, P=16):
    """img int8 [B, C_in, H, W], w int8 [D, C_in*P*P] -> int8 [B, T, D]."""
    img = _arr(img, np.int8)
    w = _arr(w, np.int8)
    mult, shift = _arr(mult, np.int32).reshape(-1), _arr(shift, np.int32).reshape(-1)
    b = None if bias is None else _arr(bias, np.int32)
    pos = _arr(pos, np.int8)
    B, C, H, W = img.shape
    D = w.shape[0]
    T = (H // P) * (W // P)
    assert w.shape[1] == C * P * P and pos.shape == (T, D)
    y = np.zeros((B, T, D), np.int8)
    lib().orc_patch_embed(_p(img, i8p), B, C, H, W, P, _p(w, i8p),
                          None if b is None else _p(b, i32p), _p(mult, i32p), _p(shift, i32p),
                          mult.shape[0], _p(pos, i8p), pos_ma, pos_mb, pos_shift, D, _p(y, i8p))
    return y


def residual_tensor(a, b, mult_a, mult_b, shift):
    a = _arr(a, np.int8)
    b = _arr(b, np.int8)
    y = np.zeros_like(a)
    lib().orc_residual_tensor(_p(a, i8p), _p(b, i8p), _p(y, i8p), a.size, mult_a,
                              mult_b, shift)
    return y


def attention(qkv, grid_h, grid_w, win_h, win_w, heads, head_dim, score_mult,
              score_shift, I0, pv_mult, pv_shift, k_inter=16, k_out=8, m_p=4,
              s_d=-1):
    qkv = _arr(qkv, np.int8)
    T, D3 = qkv.shape
    D = D3 // 3
    out = np.zeros((T, D), np.int8)
    lib().orc_attention(_p(qkv, i8p), grid_h, grid_w, win_h, win_w, D, heads,
                        head_dim, score_mult, score_shift, I0, k_inter, k_out, m_p,
                        s_d, pv_mult, pv_shift, _p(out, i8p))
    return out


_BLOCK_ARRAYS = {
    "ln1_beta": np.int32, "ln1_mult": np.int32, "ln1_shift": np.int32,
    "w_qkv": np.int8, "b_qkv": np.int32, "qkv_mult": np.int32, "qkv_shift": np.int32,
    "w_proj": np.int8, "b_proj": np.int32, "proj_mult": np.int32,
    "proj_shift": np.int32,
    "ln2_beta": np.int32, "ln2_mult": np.int32, "ln2_shift": np.int32,
    "w_fc1": np.int8, "b_fc1": np.int32, "fc1_mult": np.int32, "fc1_shift": np.int32,
    "w_fc2": np.int8, "b_fc2": np.int32, "fc2_mult": np.int32, "fc2_shift": np.int32,
}
_BLOCK_SCALARS = [
    "dim", "heads", "head_dim", "mlp_dim", "ln_iters", "score_mult", "score_shift",
    "smax_I0", "smax_k_inter", "smax_k_out", "smax_m_p", "smax_s_d", "pv_mult",
    "pv_shift", "res1_mult_a", "res1_mult_b", "res1_shift", "gelu_I0",
    "gelu_k_inter", "gelu_k_out", "gelu_mult", "gelu_shift", "res2_mult_a",
    "res2_mult_b", "res2_shift",
]


def block_struct(params: dict):
    """Build the oracle's block struct from a parameter dict.  Returns the
    struct and the list of arrays that must stay alive while it is used."""
    keep = []
    s = OrcBlock()
    for name in _BLOCK_SCALARS:
        setattr(s, name, int(params[name]))
    for name, dt in _BLOCK_ARRAYS.items():
        a = _arr(params[name], dt)
        keep.append(a)
        setattr(s, name, _p(a, i8p if dt == np.int8 else i32p))
    for stem in ("ln1", "qkv", "proj", "ln2", "fc1", "fc2"):
        setattr(s, stem + "_nq", int(np.asarray(params[stem + "_mult"]).shape[0]))
    return s, keep


def block_forward(params: dict, x, grid_h, grid_w, win_h, win_w):
    """x int8 [B, T, D] -> int8 [B, T, D]; win_h == 0 selects global attention."""
    x = _arr(x, np.int8)
    B = x.shape[0]
    y = np.zeros_like(x)
    s, keep = block_struct(params)
    lib().orc_block_forward(ctypes.byref(s), _p(x, i8p), _p(y, i8p), B, grid_h, grid_w,
                            win_h, win_w)
    del keep
    return y


def decoder_struct(params: dict):
    """Build the oracle's decoder struct from a parameter dict whose keys are
    the struct's field names (the *_nq fields are taken from the lengths of
    the multiplier arrays).  Returns the struct and the arrays to keep alive."""
    keep = []
    s = OrcDecoder()
    for name, typ in OrcDecoder._fields_:
        if name.endswith("_nq"):
            setattr(s, name, int(np.asarray(params[name[:-3] + "_mult"]).shape[0]))
        elif name == "ref_dims":  # set from the reference array by decoder_forward
            setattr(s, name, int(params.get(name, 2)))
        elif typ is c_i32:
            setattr(s, name, int(params[name]))
        else:
            a = _arr(params[name], np.int8 if typ is i8p else np.int32)
            keep.append(a)
            setattr(s, name, _p(a, typ))
    return s, keep


def decoder_forward(params: dict, tgt, memory, ref, level_hw, level_start):
    """tgt int8 [B, Q, D], memory int8 [B, S, D], ref int32 Q16 [B, Q, 2]
    (points) or [B, Q, 4] (boxes) -> int8 [B, Q, D]."""
    tgt = _arr(tgt, np.int8)
    memory = _arr(memory, np.int8)
    ref = _arr(ref, np.int32)
    level_hw = _arr(level_hw, np.int32)
    level_start = _arr(level_start, np.int32)
    B, Q, D = tgt.shape
    S = memory.shape[1]
    y = np.zeros_like(tgt)
    s, keep = decoder_struct(params)
    s.ref_dims = ref.shape[-1]
    lib().orc_decoder_forward(ctypes.byref(s), _p(tgt, i8p), _p(memory, i8p), _p(ref, i32p),
                              _p(level_hw, i32p), _p(level_start, i32p), B, Q, S, _p(y, i8p))
    del keep
    return y


def deform_nearest_index(ref_x, ref_y, off_x, off_y, H, W):
    return lib().orc_deform_nearest_index(int(ref_x), int(ref_y), int(off_x),
                                          int(off_y), int(H), int(W))


def deform_box_nearest_index(cx, cy, w, h, off_x, off_y, H, W, P):
    return lib().orc_deform_box_nearest_index(*(int(v) for v in (cx, cy, w, h, off_x, off_y,
                                                                 H, W, P)))


def deform_attn(value, level_hw, level_start, ref, offsets, logits, I0, out_mult,
                out_shift, mode=0, k_inter=16, k_out=8, m_p=4, s_d=-1):
    """value int8 [B, S, H, Dh]; ref int32 [B, Q, 2] (points) or [B, Q, 4]
    (boxes); offsets int16 [B, Q, H, L, P, 2]; logits int8 [B, Q, H, L*P]
    -> out int8 [B, Q, H*Dh]."""
    value = _arr(value, np.int8)
    level_hw = _arr(level_hw, np.int32)
    level_start = _arr(level_start, np.int32)
    ref = _arr(ref, np.int32)
    offsets = _arr(offsets, np.int16)
    logits = _arr(logits, np.int8)
    B, S, H, Dh = value.shape
    _, Q, _, L, P, _ = offsets.shape
    out = np.zeros((B, Q, H * Dh), np.int8)
    lib().orc_deform_attn(_p(value, i8p), _p(level_hw, i32p), _p(level_start, i32p),
                          L, P, _p(ref, i32p), _p(offsets, i16p), _p(logits, i8p),
                          _p(out, i8p), B, Q, H, Dh, S, I0, k_inter, k_out, m_p, s_d,
                          out_mult, out_shift, mode, ref.shape[-1])
    return out
