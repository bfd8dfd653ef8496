"""ctypes binding of libilw.so, the C ABI declared in include/ilw.h.

Argument marshalling only: every step of the computation runs in the HIP
kernels of libilw.so.  Tensors are torch tensors on a ROCm device (torch is
used for device memory and streams); calls are issued on torch's current
stream.  There is no fallback: if the library is missing or a call fails, an
IlwError is raised.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# ILW_LIBRARY_PATH loads another build of the same sources instead (the
# sanitizer run of the CPU test-suite uses a host-instrumented one).
LIB_PATH = os.environ.get("ILW_LIBRARY_PATH") or os.path.join(_HERE, "libilw.so")
ABI_VERSION = 9

c_i32, c_i64, c_vp, c_size = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t


class IlwError(RuntimeError):
    pass


class Dyadic(ctypes.Structure):
    _fields_ = [("mult", c_vp), ("shift", c_vp), ("n", c_i32)]


class AttnParams(ctypes.Structure):
    _fields_ = [("score_mult", c_i32), ("score_shift", c_i32), ("I0", c_i32),
                ("k_inter", c_i32), ("k_out", c_i32), ("m_p", c_i32), ("s_d", c_i32),
                ("pv_mult", c_i32), ("pv_shift", c_i32)]


class BlockParams(ctypes.Structure):
    _fields_ = [
        ("dim", c_i32), ("heads", c_i32), ("head_dim", c_i32), ("mlp_dim", c_i32),
        ("ln_iters", c_i32),
        ("ln1_beta", c_vp), ("ln1_out", Dyadic),
        ("w_qkv", c_vp), ("b_qkv", c_vp), ("qkv", Dyadic),
        ("attn", AttnParams),
        ("w_proj", c_vp), ("b_proj", c_vp), ("proj", Dyadic),
        ("res1_mult_a", c_i32), ("res1_mult_b", c_i32), ("res1_shift", c_i32),
        ("ln2_beta", c_vp), ("ln2_out", Dyadic),
        ("w_fc1", c_vp), ("b_fc1", c_vp), ("fc1", Dyadic),
        ("gelu_I0", c_i32), ("gelu_k_inter", c_i32), ("gelu_k_out", c_i32),
        ("gelu_mult", c_i32), ("gelu_shift", c_i32),
        ("w_fc2", c_vp), ("b_fc2", c_vp), ("fc2", Dyadic),
        ("res2_mult_a", c_i32), ("res2_mult_b", c_i32), ("res2_shift", c_i32),
    ]


def _lin(stem):
    return [("w_" + stem, c_vp), ("b_" + stem, c_vp), (stem, Dyadic)]


class DecoderParams(ctypes.Structure):
    _fields_ = (
        [(n, c_i32) for n in ("dim", "heads", "ffn_dim", "levels", "points", "ln_iters")]
        + _lin("qkv") + [("attn", AttnParams)] + _lin("o")
        + [(n, c_i32) for n in ("res1_mult_a", "res1_mult_b", "res1_shift")]
        + [("ln1_beta", c_vp), ("ln1_out", Dyadic)]
        + _lin("val") + _lin("off") + _lin("attw")
        + [(n, c_i32) for n in ("da_I0", "da_s_d", "da_out_mult", "da_out_shift", "da_mode",
                                "ref_dims")]
        + _lin("co")
        + [(n, c_i32) for n in ("res2_mult_a", "res2_mult_b", "res2_shift")]
        + [("ln2_beta", c_vp), ("ln2_out", Dyadic)]
        + _lin("fc1")
        + [(n, c_i32) for n in ("gelu_I0", "gelu_k_inter", "gelu_k_out", "gelu_mult",
                                "gelu_shift")]
        + _lin("fc2")
        + [(n, c_i32) for n in ("res3_mult_a", "res3_mult_b", "res3_shift")]
        + [("ln3_beta", c_vp), ("ln3_out", Dyadic)])


_SIGS = {
    "ilw_last_error": (ctypes.c_char_p, []),
    "ilw_abi_version": (ctypes.c_int, []),
    "ilw_linear": (ctypes.c_int, [c_vp, c_vp, c_vp, Dyadic, c_vp, c_i64, c_i32, c_i32, c_vp]),
    "ilw_shiftmax": (ctypes.c_int, [c_vp, c_vp, c_i64, c_i32, c_i32, c_i32, c_i32, c_i32,
                                    c_i32, c_vp]),
    "ilw_sdshiftgelu": (ctypes.c_int, [c_vp, c_vp, c_i64, c_i32, c_i32, c_i32, c_i32, c_i32,
                                       c_vp]),
    "ilw_shiftmax_ivit": (ctypes.c_int, [c_vp, c_vp, c_i64, c_i32, c_i32, c_i32, c_i32, c_i32,
                                         c_vp]),
    "ilw_shiftgelu_ivit": (ctypes.c_int, [c_vp, c_vp, c_i64, c_i32, c_i32, c_i32, c_i32, c_i32,
                                          c_i32, c_vp]),
    "ilw_int_layernorm": (ctypes.c_int, [c_vp, c_vp, c_i64, c_i32, c_vp, Dyadic, c_i32,
                                         c_vp]),
    "ilw_residual_add": (ctypes.c_int, [c_vp, c_vp, c_vp, c_i64, c_i32, c_i32, c_i32, c_vp]),
    "ilw_attention_workspace_bytes": (c_size, [c_i32] * 7),
    "ilw_attention": (ctypes.c_int, [c_vp, c_vp] + [c_i32] * 8 +
                      [ctypes.POINTER(AttnParams), c_vp, c_size, c_vp]),
    "ilw_block_workspace_bytes": (c_size, [ctypes.POINTER(BlockParams)] + [c_i32] * 5),
    "ilw_block_forward": (ctypes.c_int, [ctypes.POINTER(BlockParams), c_vp, c_vp] +
                          [c_i32] * 5 + [c_vp, c_size, c_vp]),
    "ilw_block_forward_noalloc": (ctypes.c_int, [ctypes.POINTER(BlockParams), c_vp, c_vp] +
                                  [c_i32] * 5 + [c_vp]),
    "ilw_encoder_workspace_bytes": (c_size, [c_vp, c_i32, c_vp, c_i32, c_i32, c_i32]),
    "ilw_encoder_forward": (ctypes.c_int, [c_vp, c_i32, c_vp, c_vp, c_vp, c_i32, c_i32, c_i32,
                                           c_vp, c_size, c_vp]),
    "ilw_split_conv": (ctypes.c_int, [c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, Dyadic, c_vp,
                                      c_i64, c_i32, c_vp]),
    "ilw_patch_embed": (ctypes.c_int, [c_vp, c_i32, c_i32, c_i32, c_i32, c_i32, c_vp, c_vp,
                                       Dyadic, c_vp, c_i32, c_i32, c_i32, c_vp, c_i32, c_vp]),
    "ilw_decoder_workspace_bytes": (c_size, [ctypes.POINTER(DecoderParams), c_i32, c_i32,
                                             c_i32]),
    "ilw_decoder_layer": (ctypes.c_int, [ctypes.POINTER(DecoderParams), c_vp, c_vp, c_vp, c_vp,
                                         c_vp, c_vp, c_i32, c_i32, c_i32, c_vp, c_size, c_vp]),
    "ilw_profile_enable": (ctypes.c_int, [ctypes.c_int]),
    "ilw_profile_read": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(c_i32), c_i32]),
    "ilw_deform_attn": (ctypes.c_int, [c_vp, c_vp, c_vp, c_i32, c_i32, c_vp, c_vp, c_vp,
                                       c_vp] + [c_i32] * 12 + [c_vp]),
    "ilw_deform_attn_boxes": (ctypes.c_int, [c_vp, c_vp, c_vp, c_i32, c_i32, c_vp, c_vp, c_vp,
                                             c_vp] + [c_i32] * 12 + [c_vp]),
}

_LIB = None


def lib():
    """Load libilw.so (raises IlwError if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise IlwError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2607_24981_amd.build`; there is no fallback")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        if L.ilw_abi_version() != ABI_VERSION:
            raise IlwError("libilw.so ABI version mismatch")
        _LIB = L
    return _LIB


def last_error() -> str:
    return lib().ilw_last_error().decode()


def _check(rc: int, name: str):
    if rc != 0:
        raise IlwError(f"{name} failed with status {rc}: {last_error()}")


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t: torch.Tensor, dtype, name: str):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise IlwError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise IlwError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise IlwError(f"{name} must be contiguous")
    return c_vp(t.data_ptr())


def _dyadic(mult: torch.Tensor, shift: torch.Tensor) -> Dyadic:
    return Dyadic(_dev(mult, torch.int32, "mult").value, _dev(shift, torch.int32, "shift").value,
                  mult.numel())


def to_device(a, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


# ------------------------------------------------------------------ operators
def ilw_linear(x, w, b, mult, shift, y=None):
    M, K = x.shape
    N = w.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.int8, device=x.device)
    rc = lib().ilw_linear(_dev(x, torch.int8, "x"), _dev(w, torch.int8, "w"),
                          _dev(b, torch.int32, "b") if b is not None else None,
                          _dyadic(mult, shift), _dev(y, torch.int8, "y"), M, N, K, _stream())
    _check(rc, "ilw_linear")
    return y


def ilw_shiftmax(x, I0, k_inter=16, k_out=8, m_p=4, s_d=-1, y=None):
    rows, cols = x.shape
    if y is None:
        y = torch.empty_like(x)
    rc = lib().ilw_shiftmax(_dev(x, torch.int8, "x"), _dev(y, torch.int8, "y"), rows, cols,
                            I0, k_inter, k_out, m_p, s_d, _stream())
    _check(rc, "ilw_shiftmax")
    return y


def ilw_sdshiftgelu(x, I0, out_mult, out_shift, k_inter=16, k_out=8, y=None):
    if y is None:
        y = torch.empty_like(x)
    rc = lib().ilw_sdshiftgelu(_dev(x, torch.int8, "x"), _dev(y, torch.int8, "y"), x.numel(),
                               I0, k_inter, k_out, out_mult, out_shift, _stream())
    _check(rc, "ilw_sdshiftgelu")
    return y


def ilw_int_layernorm(x, beta, mult, shift, newton_iters=10, y=None):
    C = x.shape[-1]
    if y is None:
        y = torch.empty_like(x)
    rc = lib().ilw_int_layernorm(_dev(x, torch.int8, "x"), _dev(y, torch.int8, "y"),
                                 x.numel() // C, C, _dev(beta, torch.int32, "beta"),
                                 _dyadic(mult, shift), newton_iters, _stream())
    _check(rc, "ilw_int_layernorm")
    return y


def ilw_residual_add(a, b, mult_a, mult_b, shift, y=None):
    if y is None:
        y = torch.empty_like(a)
    rc = lib().ilw_residual_add(_dev(a, torch.int8, "a"), _dev(b, torch.int8, "b"),
                                _dev(y, torch.int8, "y"), a.numel(), mult_a, mult_b, shift,
                                _stream())
    _check(rc, "ilw_residual_add")
    return y


def attn_params(p: dict) -> AttnParams:
    return AttnParams(int(p["score_mult"]), int(p["score_shift"]), int(p["smax_I0"]),
                      int(p.get("smax_k_inter", 16)), int(p.get("smax_k_out", 8)),
                      int(p.get("smax_m_p", 4)), int(p.get("smax_s_d", -1)),
                      int(p["pv_mult"]), int(p["pv_shift"]))


def ilw_attention(qkv, grid_h, grid_w, win_h, win_w, heads, params: dict, out=None,
                  workspace=None):
    """qkv int8 [B, T, 3D] -> out int8 [B, T, D]."""
    B, T, D3 = qkv.shape
    D = D3 // 3
    if out is None:
        out = torch.empty((B, T, D), dtype=torch.int8, device=qkv.device)
    need = lib().ilw_attention_workspace_bytes(B, grid_h, grid_w, win_h, win_w, D, D // heads)
    if need == 0 and B > 0:
        raise IlwError(f"ilw_attention_workspace_bytes: {last_error()}")
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.int8, device=qkv.device)
    ap = attn_params(params)
    rc = lib().ilw_attention(_dev(qkv, torch.int8, "qkv"), _dev(out, torch.int8, "out"), B,
                             grid_h, grid_w, win_h, win_w, D, heads, D // heads,
                             ctypes.byref(ap), _dev(workspace, torch.int8, "workspace"),
                             workspace.numel(), _stream())
    _check(rc, "ilw_attention")
    return out


class DeviceBlock:
    """Device copy of one encoder block's parameters plus its ABI struct."""

    _ARRAYS = {"ln1_beta": torch.int32, "ln1_mult": torch.int32, "ln1_shift": torch.int32,
               "w_qkv": torch.int8, "b_qkv": torch.int32, "qkv_mult": torch.int32,
               "qkv_shift": torch.int32, "w_proj": torch.int8, "b_proj": torch.int32,
               "proj_mult": torch.int32, "proj_shift": torch.int32,
               "ln2_beta": torch.int32, "ln2_mult": torch.int32, "ln2_shift": torch.int32,
               "w_fc1": torch.int8, "b_fc1": torch.int32, "fc1_mult": torch.int32,
               "fc1_shift": torch.int32, "w_fc2": torch.int8, "b_fc2": torch.int32,
               "fc2_mult": torch.int32, "fc2_shift": torch.int32}

    def __init__(self, p: dict, device="cuda"):
        self.p = p
        self.t = {k: to_device(np.asarray(p[k]), device) for k in self._ARRAYS}
        for k, dt in self._ARRAYS.items():
            assert self.t[k].dtype == dt, (k, self.t[k].dtype)
        t = self.t
        s = BlockParams()
        s.dim, s.heads, s.head_dim = int(p["dim"]), int(p["heads"]), int(p["head_dim"])
        s.mlp_dim, s.ln_iters = int(p["mlp_dim"]), int(p["ln_iters"])
        s.ln1_beta = t["ln1_beta"].data_ptr()
        s.ln1_out = _dyadic(t["ln1_mult"], t["ln1_shift"])
        s.w_qkv, s.b_qkv = t["w_qkv"].data_ptr(), t["b_qkv"].data_ptr()
        s.qkv = _dyadic(t["qkv_mult"], t["qkv_shift"])
        s.attn = attn_params(p)
        s.w_proj, s.b_proj = t["w_proj"].data_ptr(), t["b_proj"].data_ptr()
        s.proj = _dyadic(t["proj_mult"], t["proj_shift"])
        s.res1_mult_a, s.res1_mult_b = int(p["res1_mult_a"]), int(p["res1_mult_b"])
        s.res1_shift = int(p["res1_shift"])
        s.ln2_beta = t["ln2_beta"].data_ptr()
        s.ln2_out = _dyadic(t["ln2_mult"], t["ln2_shift"])
        s.w_fc1, s.b_fc1 = t["w_fc1"].data_ptr(), t["b_fc1"].data_ptr()
        s.fc1 = _dyadic(t["fc1_mult"], t["fc1_shift"])
        s.gelu_I0, s.gelu_k_inter = int(p["gelu_I0"]), int(p["gelu_k_inter"])
        s.gelu_k_out, s.gelu_mult = int(p["gelu_k_out"]), int(p["gelu_mult"])
        s.gelu_shift = int(p["gelu_shift"])
        s.w_fc2, s.b_fc2 = t["w_fc2"].data_ptr(), t["b_fc2"].data_ptr()
        s.fc2 = _dyadic(t["fc2_mult"], t["fc2_shift"])
        s.res2_mult_a, s.res2_mult_b = int(p["res2_mult_a"]), int(p["res2_mult_b"])
        s.res2_shift = int(p["res2_shift"])
        self.struct = s

    def workspace_bytes(self, B, grid_h, grid_w, win_h, win_w) -> int:
        n = lib().ilw_block_workspace_bytes(ctypes.byref(self.struct), B, grid_h, grid_w,
                                            win_h, win_w)
        if n == 0 and B > 0:
            raise IlwError(f"ilw_block_workspace_bytes: {last_error()}")
        return n


def ilw_block_forward(block: DeviceBlock, x, grid_h, grid_w, win_h, win_w, y=None,
                      workspace=None):
    """x int8 [B, T, D] -> y int8 [B, T, D] (y may be x)."""
    B = x.shape[0]
    if y is None:
        y = torch.empty_like(x)
    if workspace is None:
        n = block.workspace_bytes(B, grid_h, grid_w, win_h, win_w)
        workspace = torch.empty(max(n, 16), dtype=torch.int8, device=x.device)
    rc = lib().ilw_block_forward(ctypes.byref(block.struct), _dev(x, torch.int8, "x"),
                                 _dev(y, torch.int8, "y"), B, grid_h, grid_w, win_h, win_w,
                                 _dev(workspace, torch.int8, "workspace"), workspace.numel(),
                                 _stream())
    _check(rc, "ilw_block_forward")
    return y


def ilw_block_forward_noalloc(block: DeviceBlock, x, grid_h, grid_w, win_h, win_w, y=None):
    """ilw_block_forward on the library's static device scratch (no workspace
    argument; the library allocates nothing).  y must be given by callers
    that cannot allocate."""
    B = x.shape[0]
    if y is None:
        y = torch.empty_like(x)
    rc = lib().ilw_block_forward_noalloc(ctypes.byref(block.struct), _dev(x, torch.int8, "x"),
                                         _dev(y, torch.int8, "y"), B, grid_h, grid_w, win_h,
                                         win_w, _stream())
    _check(rc, "ilw_block_forward_noalloc")
    return y


NOALLOC_SCRATCH_BYTES = 32 << 20


class Encoder:
    """A stack of integer encoder blocks run by ilw_encoder_forward."""

    def __init__(self, blocks: list, windows: list, grid_h: int, grid_w: int,
                 device="cuda"):
        self.blocks = [b if isinstance(b, DeviceBlock) else DeviceBlock(b, device)
                       for b in blocks]
        self.windows = [tuple(int(v) for v in w) for w in windows]
        assert len(self.windows) == len(self.blocks)
        self.grid_h, self.grid_w = grid_h, grid_w
        self.device = device
        n = len(self.blocks)
        self._structs = (BlockParams * n)(*[b.struct for b in self.blocks])
        self._win = np.ascontiguousarray(np.asarray(self.windows, np.int32).reshape(n, 2))
        self._ws = None

    def workspace_bytes(self, B) -> int:
        n = lib().ilw_encoder_workspace_bytes(ctypes.addressof(self._structs), len(self.blocks),
                                              self._win.ctypes.data_as(c_vp), B, self.grid_h,
                                              self.grid_w)
        if n == 0 and B > 0:
            raise IlwError(f"ilw_encoder_workspace_bytes: {last_error()}")
        return n

    def workspace(self, B):
        need = self.workspace_bytes(B)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(max(need, 16), dtype=torch.int8, device=self.device)
        return self._ws

    def forward(self, x, out=None, workspace=None):
        """x int8 [B, T, D] -> int8 [B, T, D] (out may be x)."""
        ws = self.workspace(x.shape[0]) if workspace is None else workspace
        if out is None:
            out = torch.empty_like(x)
        rc = lib().ilw_encoder_forward(ctypes.addressof(self._structs), len(self.blocks),
                                       self._win.ctypes.data_as(c_vp),
                                       _dev(x, torch.int8, "x"), _dev(out, torch.int8, "out"),
                                       x.shape[0], self.grid_h, self.grid_w,
                                       _dev(ws, torch.int8, "workspace"), ws.numel(),
                                       _stream())
        _check(rc, "ilw_encoder_forward")
        return out

    def forward_streams(self, x, out, parts: int):
        """The batch split into `parts` image ranges, each run on its own
        stream (forked from and joined back into the current stream), so that
        one part's attention shares the GPU with another part's linears.
        Each part has its own workspace.  Capturable into a HIP graph."""
        B = x.shape[0]
        bounds = [B * i // parts for i in range(parts + 1)]
        if getattr(self, "_part_streams", None) is None or len(self._part_streams) != parts:
            self._part_streams = [torch.cuda.Stream(device=x.device) for _ in range(parts)]
            self._part_ws = [None] * parts
        cur = torch.cuda.current_stream(x.device)
        for i, st in enumerate(self._part_streams):
            nb = bounds[i + 1] - bounds[i]
            need = max(self.workspace_bytes(nb), 16)
            if self._part_ws[i] is None or self._part_ws[i].numel() < need:
                self._part_ws[i] = torch.empty(need, dtype=torch.int8, device=x.device)
            st.wait_stream(cur)
        for i, st in enumerate(self._part_streams):
            b0, b1 = bounds[i], bounds[i + 1]
            if b1 > b0:
                with torch.cuda.stream(st):
                    self.forward(x[b0:b1], out[b0:b1], workspace=self._part_ws[i])
        for st in self._part_streams:
            cur.wait_stream(st)
        return out


def ilw_patch_embed(img, w, bias, mult, shift, pos, pos_mult_a, pos_mult_b, pos_shift,
                    patch=16, y=None):
    """img int8 [B, C, H, W], w int8 [D, C*16*16] -> int8 [B, T, D] with the
    positional embedding pos int8 [T, D] added."""
    B, C, H, W = img.shape
    D = w.shape[0]
    T = (H // patch) * (W // patch)
    if y is None:
        y = torch.empty((B, T, D), dtype=torch.int8, device=img.device)
    rc = lib().ilw_patch_embed(_dev(img, torch.int8, "img"), B, C, H, W, patch,
                               _dev(w, torch.int8, "w"),
                               None if bias is None else _dev(bias, torch.int32, "bias"),
                               _dyadic(mult, shift), _dev(pos, torch.int8, "pos"), pos_mult_a,
                               pos_mult_b, pos_shift, _dev(y, torch.int8, "y"), D, _stream())
    _check(rc, "ilw_patch_embed")
    return y


def ilw_shiftmax_ivit(x, I0, M=31, k_inter=16, k_out=8, y=None):
    """I-ViT Shiftmax (fixed division precision M) of every row of int8 x."""
    cols = x.shape[-1]
    rows = x.numel() // cols
    if y is None:
        y = torch.empty_like(x)
    _check(lib().ilw_shiftmax_ivit(_dev(x, torch.int8, "x"), _dev(y, torch.int8, "y"), rows,
                                   cols, I0, k_inter, k_out, M, _stream()), "ilw_shiftmax_ivit")
    return y


def ilw_shiftgelu_ivit(x, I0, out_mult, out_shift, k_inter=16, k_out=8, y=None):
    """I-ViT ShiftGELU (row-maximum shift) of every row of int8 x, requantized."""
    cols = x.shape[-1]
    rows = x.numel() // cols
    if y is None:
        y = torch.empty_like(x)
    _check(lib().ilw_shiftgelu_ivit(_dev(x, torch.int8, "x"), _dev(y, torch.int8, "y"), rows,
                                    cols, I0, k_inter, k_out, out_mult, out_shift, _stream()),
           "ilw_shiftgelu_ivit")
    return y


class DeviceDecoder:
    """Device copy of one decoder layer's parameters plus its ABI struct.
    `p` is the parameter dict of the oracle's decoder (same keys)."""

    def __init__(self, p: dict, device="cuda"):
        self.p = p
        self.t = {}
        for k, v in p.items():
            if isinstance(v, np.ndarray):
                self.t[k] = to_device(v, device)
        s = DecoderParams()
        for n in ("dim", "heads", "ffn_dim", "levels", "points", "ln_iters", "da_I0", "da_s_d",
                  "da_out_mult", "da_out_shift", "da_mode", "gelu_I0", "gelu_k_inter",
                  "gelu_k_out", "gelu_mult", "gelu_shift", "res1_mult_a", "res1_mult_b",
                  "res1_shift", "res2_mult_a", "res2_mult_b", "res2_shift", "res3_mult_a",
                  "res3_mult_b", "res3_shift"):
            setattr(s, n, int(p[n]))
        s.ref_dims = int(p.get("ref_dims", 2))
        for stem in ("qkv", "o", "val", "off", "attw", "co", "fc1", "fc2"):
            setattr(s, "w_" + stem, self.t["w_" + stem].data_ptr())
            setattr(s, "b_" + stem, self.t["b_" + stem].data_ptr())
            setattr(s, stem, _dyadic(self.t[stem + "_mult"], self.t[stem + "_shift"]))
        for stem in ("ln1", "ln2", "ln3"):
            setattr(s, stem + "_beta", self.t[stem + "_beta"].data_ptr())
            setattr(s, stem + "_out", _dyadic(self.t[stem + "_mult"], self.t[stem + "_shift"]))
        s.attn = attn_params(p)
        self.struct = s

    def workspace_bytes(self, B, Q, S) -> int:
        n = lib().ilw_decoder_workspace_bytes(ctypes.byref(self.struct), B, Q, S)
        if n == 0 and B > 0:
            raise IlwError(f"ilw_decoder_workspace_bytes: {last_error()}")
        return n


def ilw_decoder_layer(dec: DeviceDecoder, tgt, memory, ref, level_hw, level_start, y=None,
                      workspace=None):
    """tgt int8 [B, Q, D], memory int8 [B, S, D], ref int32 [B, Q, 2] (points)
    or [B, Q, 4] (boxes, as the layer's ref_dims says); level_hw / level_start
    host arrays -> int8 [B, Q, D]."""
    B, Q, D = tgt.shape
    S = memory.shape[1]
    rd = dec.struct.ref_dims
    if tuple(ref.shape) != (B, Q, rd):
        raise ValueError(f"ref has shape {tuple(ref.shape)}, expected {(B, Q, rd)}")
    L = dec.p["levels"]
    hw = np.ascontiguousarray(np.asarray(level_hw, np.int32).reshape(L, 2))
    st = np.ascontiguousarray(np.asarray(level_start, np.int32).reshape(L))
    if y is None:
        y = torch.empty_like(tgt)
    if workspace is None:
        workspace = torch.empty(max(dec.workspace_bytes(B, Q, S), 16), dtype=torch.int8,
                                device=tgt.device)
    rc = lib().ilw_decoder_layer(ctypes.byref(dec.struct), _dev(tgt, torch.int8, "tgt"),
                                 _dev(memory, torch.int8, "memory"),
                                 _dev(ref, torch.int32, "ref"), hw.ctypes.data_as(c_vp),
                                 st.ctypes.data_as(c_vp), _dev(y, torch.int8, "y"), B, Q, S,
                                 _dev(workspace, torch.int8, "workspace"), workspace.numel(),
                                 _stream())
    _check(rc, "ilw_decoder_layer")
    return y


def ilw_split_conv(xs, ws, branch_mults, branch_shifts, bias, out_mult, out_shift, y=None):
    """Scale-preserving split convolution: xs[b] int8 [M, C_b], ws[b] int8
    [N, C_b], per-branch rescale dyadics, bias int32 [N] or None, output
    dyadic -> int8 [M, N]."""
    nb = len(xs)
    assert len(ws) == len(branch_mults) == len(branch_shifts) == nb
    M, N = xs[0].shape[0], ws[0].shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.int8, device=xs[0].device)
    xp = (c_vp * nb)(*[_dev(x, torch.int8, "x") for x in xs])
    wp = (c_vp * nb)(*[_dev(w, torch.int8, "w") for w in ws])
    ch = (c_i32 * nb)(*[int(x.shape[1]) for x in xs])
    br = (Dyadic * nb)(*[_dyadic(m, s_) for m, s_ in zip(branch_mults, branch_shifts)])
    rc = lib().ilw_split_conv(nb, xp, ch, wp, br,
                              None if bias is None else _dev(bias, torch.int32, "bias"),
                              _dyadic(out_mult, out_shift), _dev(y, torch.int8, "y"), M, N,
                              _stream())
    _check(rc, "ilw_split_conv")
    return y


def _deform(entry, ref_dims, value, level_hw, level_start, ref, offsets, logits, I0, out_mult,
            out_shift, mode, s_d, out, k_inter, k_out, m_p):
    B, S, H, Dh = value.shape
    _, Q, _, L, P, _ = offsets.shape
    if tuple(ref.shape) != (B, Q, ref_dims):
        raise ValueError(f"ref has shape {tuple(ref.shape)}, expected {(B, Q, ref_dims)}")
    hw = np.ascontiguousarray(np.asarray(level_hw, np.int32).reshape(L, 2))
    st = np.ascontiguousarray(np.asarray(level_start, np.int32).reshape(L))
    if out is None:
        out = torch.empty((B, Q, H * Dh), dtype=torch.int8, device=value.device)
    rc = getattr(lib(), entry)(_dev(value, torch.int8, "value"),
                               hw.ctypes.data_as(c_vp), st.ctypes.data_as(c_vp), L, P,
                               _dev(ref, torch.int32, "ref"),
                               _dev(offsets, torch.int16, "offsets"),
                               _dev(logits, torch.int8, "logits"), _dev(out, torch.int8, "out"),
                               B, Q, H, Dh, I0, k_inter, k_out, m_p, s_d, out_mult,
                               out_shift, mode, _stream())
    _check(rc, entry)
    return out


def ilw_deform_attn(value, level_hw, level_start, ref, offsets, logits, I0, out_mult,
                    out_shift, mode=0, s_d=-1, out=None, k_inter=16, k_out=8, m_p=4):
    """value int8 [B, S, H, Dh]; ref int32 [B, Q, 2] (points); offsets int16
    [B, Q, H, L, P, 2]; logits int8 [B, Q, H, L*P]; level_hw / level_start are
    host arrays; I0, k_inter, k_out, m_p, s_d are the Constrained Shiftmax
    parameters of the sampling weights."""
    return _deform("ilw_deform_attn", 2, value, level_hw, level_start, ref, offsets, logits,
                   I0, out_mult, out_shift, mode, s_d, out, k_inter, k_out, m_p)


def ilw_deform_attn_boxes(value, level_hw, level_start, ref, offsets, logits, I0, out_mult,
                          out_shift, mode=0, s_d=-1, out=None, k_inter=16, k_out=8, m_p=4):
    """As ilw_deform_attn with reference boxes: ref int32 [B, Q, 4]
    (cx, cy, w, h), offsets in Q8 units of size / (2 P)."""
    return _deform("ilw_deform_attn_boxes", 4, value, level_hw, level_start, ref, offsets,
                   logits, I0, out_mult, out_shift, mode, s_d, out, k_inter, k_out, m_p)


STAGES = ["layernorm", "gemm_qkv", "attention", "gemm_proj", "gemm_fc1", "gemm_fc2",
          "relayout", "deform", "block_tail", "split_conv", "patch_embed", "decoder", "tail384"]


def profile_enable(on: bool = True):
    _check(lib().ilw_profile_enable(1 if on else 0), "ilw_profile_enable")


def profile_read() -> dict:
    """{stage: (total kernel ms, launches)} of the launches since enabling."""
    n = len(STAGES)
    ms = (ctypes.c_double * n)()
    cnt = (c_i32 * n)()
    _check(lib().ilw_profile_read(ms, cnt, n), "ilw_profile_read")
    return {STAGES[i]: (ms[i], cnt[i]) for i in range(n)}
