"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/ilw.h declares, and rejects invalid arguments with the
documented status before anything is launched."""
import ctypes
import os
import re

import pytest

from paper_2607_24981_amd import ilw

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ilw.h")

OK, E_NULL, E_SHAPE, E_PARAM, E_UNSUP, E_WS, E_HIP = 0, -1, -2, -3, -4, -5, -6
FAKE = 0x10000  # aligned, never dereferenced: every call below fails validation


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ilw_\w+)\s*\(", text)))


def test_header_declares_the_paper_operators():
    names = declared_functions()
    for n in ("ilw_block_forward", "ilw_shiftmax", "ilw_sdshiftgelu", "ilw_int_layernorm",
              "ilw_deform_attn"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = ctypes.CDLL(ilw.LIB_PATH)
    for name in declared_functions():
        assert hasattr(L, name), name
    assert set(ilw._SIGS) == set(declared_functions())


def test_abi_version_and_error_text():
    L = ilw.lib()
    assert L.ilw_abi_version() == ilw.ABI_VERSION
    rc = L.ilw_shiftmax(None, None, 4, 0, 16, 16, 8, 4, -1, None)
    assert rc == E_SHAPE
    assert "cols" in ilw.last_error()


@pytest.mark.parametrize("args,code", [
    ((FAKE, FAKE, 4, 0, 16, 16, 8, 4, -1), E_SHAPE),      # empty rows
    ((FAKE, FAKE, 4, 70000, 16, 16, 8, 4, -1), E_SHAPE),  # cols too long
    ((FAKE, FAKE, -1, 8, 16, 16, 8, 4, -1), E_SHAPE),
    ((FAKE, FAKE, 4, 8, 0, 16, 8, 4, -1), E_PARAM),       # I0
    ((FAKE, FAKE, 4, 8, 1 << 14, 16, 8, 4, -1), E_PARAM),
    ((FAKE, FAKE, 4, 8, 16, 17, 8, 4, -1), E_PARAM),      # k_inter
    ((FAKE, FAKE, 4, 8, 16, 16, 9, 4, -1), E_PARAM),      # k_out
    ((FAKE, FAKE, 4, 8, 16, 16, 8, 32, -1), E_PARAM),     # m_p
    ((FAKE, FAKE, 4, 8, 16, 16, 8, 4, -2), E_PARAM),      # s_d
    ((FAKE, FAKE, 4, 8, 16, 16, 8, 4, 32), E_PARAM),
    ((None, FAKE, 4, 8, 16, 16, 8, 4, -1), E_NULL),
    ((FAKE, FAKE, 0, 8, 16, 16, 8, 4, -1), OK),           # empty: no launch
])
def test_shiftmax_validation(args, code):
    assert ilw.lib().ilw_shiftmax(*args, None) == code


def test_linear_validation():
    L = ilw.lib()
    d = ilw.Dyadic(FAKE, FAKE, 32)
    assert L.ilw_linear(FAKE, FAKE, None, d, FAKE, 10, 30, 64, None) == E_SHAPE   # N % 16
    assert L.ilw_linear(FAKE, FAKE, None, d, FAKE, 10, 32, 40, None) == E_SHAPE   # K % 16
    assert L.ilw_linear(FAKE + 4, FAKE, None, d, FAKE, 10, 32, 64, None) == E_PARAM
    assert L.ilw_linear(None, FAKE, None, d, FAKE, 10, 32, 64, None) == E_NULL
    assert L.ilw_linear(FAKE, FAKE, None, ilw.Dyadic(FAKE, FAKE, 7), FAKE, 10, 32, 64,
                        None) == E_SHAPE
    assert L.ilw_linear(FAKE, FAKE, None, ilw.Dyadic(None, FAKE, 1), FAKE, 10, 32, 64,
                        None) == E_NULL
    assert L.ilw_linear(FAKE, FAKE, None, d, FAKE, 0, 32, 64, None) == OK


def test_elementwise_and_layernorm_validation():
    L = ilw.lib()
    assert L.ilw_sdshiftgelu(FAKE, FAKE, 10, 0, 16, 8, 1 << 30, 36, None) == E_PARAM
    assert L.ilw_sdshiftgelu(FAKE, FAKE, 10, 16, 16, 8, 1 << 30, 63, None) == E_PARAM
    assert L.ilw_sdshiftgelu(FAKE + 1, FAKE, 10, 16, 16, 8, 1 << 30, 36, None) == E_PARAM
    assert L.ilw_residual_add(FAKE, FAKE, FAKE, 10, 1, 1, 0, None) == E_PARAM
    assert L.ilw_residual_add(FAKE, FAKE, FAKE, 10, -2 ** 31, 1, 3, None) == E_PARAM
    d = ilw.Dyadic(FAKE, FAKE, 192)
    assert L.ilw_int_layernorm(FAKE, FAKE, 5, 190, FAKE, d, 10, None) == E_SHAPE
    assert L.ilw_int_layernorm(FAKE, FAKE, 5, 192, FAKE, d, 0, None) == E_PARAM
    assert L.ilw_int_layernorm(FAKE, FAKE, 5, 192, None, d, 10, None) == E_NULL
    assert L.ilw_int_layernorm(FAKE, FAKE, 5, 192, FAKE, ilw.Dyadic(FAKE, FAKE, 3), 10,
                               None) == E_SHAPE


def _block_struct(**over):
    s = ilw.BlockParams()
    s.dim, s.heads, s.head_dim, s.mlp_dim, s.ln_iters = 192, 3, 64, 768, 10
    for f in ("ln1_beta", "ln2_beta", "w_qkv", "b_qkv", "w_proj", "b_proj", "w_fc1",
              "b_fc1", "w_fc2", "b_fc2"):
        setattr(s, f, FAKE)
    s.ln1_out = s.ln2_out = ilw.Dyadic(FAKE, FAKE, 192)
    s.qkv = ilw.Dyadic(FAKE, FAKE, 576)
    s.proj = s.fc2 = ilw.Dyadic(FAKE, FAKE, 1)
    s.fc1 = ilw.Dyadic(FAKE, FAKE, 768)
    s.attn = ilw.AttnParams(1 << 30, 36, 16, 16, 8, 4, -1, 1 << 30, 36)
    s.res1_mult_a = s.res1_mult_b = s.res2_mult_a = s.res2_mult_b = 1 << 30
    s.res1_shift = s.res2_shift = 31
    s.gelu_I0, s.gelu_k_inter, s.gelu_k_out = 16, 16, 8
    s.gelu_mult, s.gelu_shift = 1 << 30, 36
    for k, v in over.items():
        setattr(s, k, v)
    return s


def test_block_workspace_and_validation():
    L = ilw.lib()
    s = _block_struct()
    n = L.ilw_block_workspace_bytes(ctypes.byref(s), 2, 40, 40, 20, 20)
    # LN out, Q, K, V^T, attention out, x1 (D each per token) and the MLP hidden
    assert n >= 2 * 1600 * (6 * 192 + 768)
    assert L.ilw_block_workspace_bytes(ctypes.byref(s), 2, 40, 40, 0, 0) >= 2 * 1600 * (6 * 192 + 768)
    bad = [
        (_block_struct(head_dim=32, heads=6), E_UNSUP),
        (_block_struct(dim=190), E_SHAPE),
        (_block_struct(mlp_dim=770), E_SHAPE),
        (_block_struct(ln_iters=0), E_PARAM),
        (_block_struct(w_fc2=None), E_NULL),
        (_block_struct(w_fc2=FAKE + 8), E_PARAM),
        (_block_struct(qkv=ilw.Dyadic(FAKE, FAKE, 192)), E_SHAPE),
        (_block_struct(attn=ilw.AttnParams(1 << 30, 0, 16, 16, 8, 4, -1, 1 << 30, 36)),
         E_PARAM),
        (_block_struct(gelu_I0=0), E_PARAM),
        (_block_struct(res2_shift=63), E_PARAM),
    ]
    for st, code in bad:
        assert L.ilw_block_workspace_bytes(ctypes.byref(st), 2, 40, 40, 20, 20) == 0
        rc = L.ilw_block_forward(ctypes.byref(st), FAKE, FAKE, 2, 40, 40, 20, 20, FAKE,
                                 1 << 30, None)
        assert rc == code, (rc, code, ilw.last_error())
    # geometry: windows must tile the grid; window token limit
    assert L.ilw_block_forward(ctypes.byref(s), FAKE, FAKE, 2, 40, 40, 30, 30, FAKE, n,
                               None) == E_SHAPE
    assert L.ilw_block_forward(ctypes.byref(s), FAKE, FAKE, 2, 64, 64, 0, 0, FAKE, 1 << 30,
                               None) == E_UNSUP
    # workspace too small / missing
    assert L.ilw_block_forward(ctypes.byref(s), FAKE, FAKE, 2, 40, 40, 20, 20, FAKE, n - 1,
                               None) == E_WS
    assert L.ilw_block_forward(ctypes.byref(s), FAKE, FAKE, 2, 40, 40, 20, 20, None, n,
                               None) == E_WS
    assert L.ilw_block_forward(ctypes.byref(s), FAKE, FAKE, 0, 40, 40, 20, 20, None, 0,
                               None) == OK


def test_encoder_workspace_and_validation():
    L = ilw.lib()
    blocks = (ilw.BlockParams * 3)(_block_struct(), _block_struct(), _block_struct())
    win = (ctypes.c_int32 * 6)(20, 20, 0, 0, 20, 20)
    n = L.ilw_encoder_workspace_bytes(blocks, 3, win, 2, 40, 40)
    one = max(L.ilw_block_workspace_bytes(ctypes.byref(_block_struct()), 2, 40, 40, w, w)
              for w in (0, 20))
    assert n >= one  # the Q K V^T region is sized for the largest block
    assert L.ilw_encoder_forward(blocks, 3, win, FAKE, FAKE, 2, 40, 40, FAKE, n - 1,
                                 None) == E_WS
    assert L.ilw_encoder_forward(blocks, 3, None, FAKE, FAKE, 2, 40, 40, FAKE, n,
                                 None) == E_NULL
    assert L.ilw_encoder_forward(blocks, 0, win, FAKE, FAKE, 2, 40, 40, FAKE, n,
                                 None) == E_SHAPE
    assert L.ilw_encoder_forward(blocks, 3, win, FAKE, FAKE, 0, 40, 40, None, 0, None) == OK
    # every block is validated; the residual width must not change
    mixed = (ilw.BlockParams * 2)(_block_struct(),
                                  _block_struct(dim=384, heads=6,
                                                ln1_out=ilw.Dyadic(FAKE, FAKE, 384),
                                                ln2_out=ilw.Dyadic(FAKE, FAKE, 384),
                                                qkv=ilw.Dyadic(FAKE, FAKE, 1152)))
    assert L.ilw_encoder_forward(mixed, 2, win, FAKE, FAKE, 2, 40, 40, FAKE, 1 << 30,
                                 None) == E_SHAPE
    assert "residual stream" in ilw.last_error()
    bad = (ilw.BlockParams * 2)(_block_struct(), _block_struct(gelu_I0=0))
    assert L.ilw_encoder_forward(bad, 2, win, FAKE, FAKE, 2, 40, 40, FAKE, 1 << 30,
                                 None) == E_PARAM
    badwin = (ctypes.c_int32 * 4)(20, 20, 30, 30)
    assert L.ilw_encoder_forward(blocks, 2, badwin, FAKE, FAKE, 2, 40, 40, FAKE, 1 << 30,
                                 None) == E_SHAPE


def test_attention_and_deform_validation():
    L = ilw.lib()
    ap = ilw.AttnParams(1 << 30, 36, 16, 16, 8, 4, -1, 1 << 30, 36)
    ws = L.ilw_attention_workspace_bytes(1, 16, 16, 0, 0, 192, 64)
    assert L.ilw_attention_workspace_bytes(1, 16, 16, 0, 0, 192, 32) == 2 * ws
    assert L.ilw_attention_workspace_bytes(1, 16, 16, 0, 0, 192, 48) == 0
    assert ws >= 3 * 256 * 192
    assert L.ilw_attention(FAKE, FAKE, 1, 16, 16, 0, 0, 192, 12, 16, ctypes.byref(ap), FAKE,
                           ws, None) == E_UNSUP
    assert L.ilw_attention(FAKE, FAKE, 1, 16, 16, 0, 0, 192, 3, 64, ctypes.byref(ap), FAKE,
                           ws - 1, None) == E_WS
    assert L.ilw_attention(FAKE, FAKE, 1, 16, 16, 0, 0, 192, 3, 64, None, FAKE, ws,
                           None) == E_NULL
    hw = (ctypes.c_int32 * 6)(80, 80, 40, 40, 20, 20)
    st = (ctypes.c_int32 * 3)(0, 6400, 8000)
    args = dict(L=3, P=4, B=8, Q=300, heads=8, head_dim=32, I0=16, k_inter=16, k_out=8,
                m_p=4, s_d=-1, m=1 << 30, s=34, mode=0)

    def call(**o):
        a = {**args, **o}
        return L.ilw_deform_attn(FAKE, hw, st, a["L"], a["P"], FAKE, FAKE, FAKE, FAKE, a["B"],
                                 a["Q"], a["heads"], a["head_dim"], a["I0"], a["k_inter"],
                                 a["k_out"], a["m_p"], a["s_d"], a["m"], a["s"], a["mode"], None)
    assert call(mode=2) == E_PARAM
    assert call(head_dim=30) == E_SHAPE
    assert call(P=30) == E_SHAPE
    assert call(I0=0) == E_PARAM
    assert call(k_inter=17) == E_PARAM
    assert call(k_out=9) == E_PARAM
    assert call(k_out=1) == E_PARAM
    assert call(m_p=32) == E_PARAM
    assert call(s_d=32) == E_PARAM
    assert call(mode=1, s=50) == E_PARAM
    assert call(Q=0) == OK
    assert L.ilw_deform_attn(FAKE, None, st, 3, 4, FAKE, FAKE, FAKE, FAKE, 8, 300, 8, 32, 16,
                             16, 8, 4, -1, 1 << 30, 34, 0, None) == E_NULL


def test_split_conv_validation():
    L = ilw.lib()
    d = ilw.Dyadic(FAKE, FAKE, 1)

    def call(nb=2, chans=(64, 128), N=64, M=10, br=None, out=None, x=True, w=True, y=FAKE):
        xp = (ctypes.c_void_p * max(nb, 1))(*([FAKE] * max(nb, 1)))
        wp = (ctypes.c_void_p * max(nb, 1))(*([FAKE] * max(nb, 1)))
        ch = (ctypes.c_int32 * max(nb, 1))(*(list(chans) + [64] * max(nb, 1))[:max(nb, 1)])
        bd = br if br is not None else (ilw.Dyadic * max(nb, 1))(*([d] * max(nb, 1)))
        return L.ilw_split_conv(nb, xp if x else None, ch, wp if w else None, bd, None,
                                out if out is not None else d, y, M, N, None)

    assert call(nb=0) == E_SHAPE
    assert call(nb=9, chans=(64,) * 9) == E_SHAPE
    assert call(chans=(64, 100)) == E_SHAPE          # not a multiple of 64
    assert call(chans=(64, 65600)) == E_SHAPE
    assert call(N=40) == E_SHAPE                     # N % 16
    assert call(x=False) == E_NULL
    assert call(w=False) == E_NULL
    assert call(br=(ilw.Dyadic * 2)(d, ilw.Dyadic(FAKE, FAKE, 7))) == E_SHAPE
    assert call(br=(ilw.Dyadic * 2)(d, ilw.Dyadic(None, FAKE, 1))) == E_NULL
    assert call(out=ilw.Dyadic(FAKE, FAKE, 3)) == E_SHAPE
    assert call(M=0) == OK
    assert call(y=FAKE + 2) == E_PARAM


def test_ivit_baseline_validation():
    L = ilw.lib()
    assert L.ilw_shiftmax_ivit(FAKE, FAKE, 4, 8, 16, 16, 8, 7, None) == E_PARAM   # M < k_out
    assert L.ilw_shiftmax_ivit(FAKE, FAKE, 4, 8, 16, 16, 8, 33, None) == E_PARAM
    assert L.ilw_shiftmax_ivit(FAKE, FAKE, 4, 0, 16, 16, 8, 31, None) == E_SHAPE
    assert L.ilw_shiftmax_ivit(FAKE, FAKE, 4, 8, 0, 16, 8, 31, None) == E_PARAM
    assert L.ilw_shiftmax_ivit(None, FAKE, 4, 8, 16, 16, 8, 31, None) == E_NULL
    assert L.ilw_shiftmax_ivit(FAKE, FAKE, 0, 8, 16, 16, 8, 31, None) == OK
    assert L.ilw_shiftgelu_ivit(FAKE, FAKE, 4, 8, 16, 16, 8, 1 << 30, 63, None) == E_PARAM
    assert L.ilw_shiftgelu_ivit(FAKE, FAKE, 4, 70000, 16, 16, 8, 1 << 30, 36, None) == E_SHAPE
    assert L.ilw_shiftgelu_ivit(FAKE, None, 4, 8, 16, 16, 8, 1 << 30, 36, None) == E_NULL
