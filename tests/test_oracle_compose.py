"""Pins of the oracle's composed operators: attention, the encoder block and
the deformable sampling core.

Attention is checked against numpy matmuls with windows cut by numpy
reshapes; the block against the chain of separately pinned operators; the
sampling locations against torch's grid_sample (nearest and bilinear, zero
padding, half-pixel convention) on the CPU.
"""
import math

import numpy as np
import pytest
import torch

from paper_2607_24981_amd import synth


def np_requant(v, m, s):
    v = v.astype(np.int64) * np.int64(m) + (np.int64(1) << np.int64(s - 1))
    return np.clip(v >> np.int64(s), -127, 127).astype(np.int8)


def window_token_ids(gh, gw, wh, ww):
    """[n_windows, wh*ww] token ids, cut from the grid with numpy reshapes."""
    if wh == 0:
        return np.arange(gh * gw).reshape(1, -1)
    ids = np.arange(gh * gw).reshape(gh // wh, wh, gw // ww, ww)
    return ids.transpose(0, 2, 1, 3).reshape(-1, wh * ww)


def np_attention(orc, qkv, gh, gw, wh, ww, heads, dh, p):
    T, D3 = qkv.shape
    D = D3 // 3
    out = np.zeros((T, D), np.int8)
    for ids in window_token_ids(gh, gw, wh, ww):
        for h in range(heads):
            q = qkv[ids, h * dh:(h + 1) * dh].astype(np.int64)
            k = qkv[ids, D + h * dh:D + (h + 1) * dh].astype(np.int64)
            v = qkv[ids, 2 * D + h * dh:2 * D + (h + 1) * dh].astype(np.int64)
            s8 = np_requant(q @ k.T, p["score_mult"], p["score_shift"])
            P = orc.shiftmax_rows(s8, p["smax_I0"]).astype(np.int64)
            out[ids, h * dh:(h + 1) * dh] = np_requant(P @ v, p["pv_mult"], p["pv_shift"])
    return out


@pytest.mark.parametrize("grid,win", [((8, 8), (0, 0)), ((8, 8), (4, 4)),
                                      ((6, 10), (3, 5)), ((5, 5), (0, 0))])
def test_attention_against_numpy(orc, grid, win):
    rng = np.random.default_rng(3)
    heads, dh = 2, 16
    D = heads * dh
    T = grid[0] * grid[1]
    qkv = rng.integers(-127, 128, (T, 3 * D)).astype(np.int8)
    p = {"score_mult": 1 << 30, "score_shift": 36, "smax_I0": 24,
         "pv_mult": 1 << 30, "pv_shift": 36}
    ref = np_attention(orc, qkv, grid[0], grid[1], win[0], win[1], heads, dh, p)
    got = orc.attention(qkv, grid[0], grid[1], win[0], win[1], heads, dh,
                        p["score_mult"], p["score_shift"], p["smax_I0"],
                        p["pv_mult"], p["pv_shift"])
    assert np.array_equal(got, ref)


def test_window_attention_is_global_attention_per_window(orc):
    rng = np.random.default_rng(4)
    heads, dh, gh, gw, wh, ww = 2, 8, 8, 12, 4, 6
    D = heads * dh
    qkv = rng.integers(-127, 128, (gh * gw, 3 * D)).astype(np.int8)
    args = (heads, dh, 1 << 30, 35, 16, 1 << 30, 35)
    win = orc.attention(qkv, gh, gw, wh, ww, *args)
    for ids in window_token_ids(gh, gw, wh, ww):
        sub = orc.attention(qkv[ids], wh, ww, 0, 0, *args)
        assert np.array_equal(win[ids], sub)


def chain_block(orc, p, x, gh, gw, wh, ww):
    """The block as the chain of separately pinned oracle operators."""
    out = []
    for xb in x:
        h = orc.int_layernorm(xb, p["ln1_beta"], p["ln1_mult"], p["ln1_shift"], p["ln_iters"])
        qkv = orc.linear(h, p["w_qkv"], p["b_qkv"], p["qkv_mult"], p["qkv_shift"])
        a = orc.attention(qkv, gh, gw, wh, ww, p["heads"], p["head_dim"], p["score_mult"],
                          p["score_shift"], p["smax_I0"], p["pv_mult"], p["pv_shift"])
        pr = orc.linear(a, p["w_proj"], p["b_proj"], p["proj_mult"], p["proj_shift"])
        x1 = orc.residual_tensor(pr, xb, p["res1_mult_a"], p["res1_mult_b"], p["res1_shift"])
        h2 = orc.int_layernorm(x1, p["ln2_beta"], p["ln2_mult"], p["ln2_shift"], p["ln_iters"])
        f1 = orc.linear(h2, p["w_fc1"], p["b_fc1"], p["fc1_mult"], p["fc1_shift"])
        g = orc.sdshiftgelu_tensor(f1, p["gelu_I0"], p["gelu_mult"], p["gelu_shift"])
        f2 = orc.linear(g, p["w_fc2"], p["b_fc2"], p["fc2_mult"], p["fc2_shift"])
        out.append(orc.residual_tensor(f2, x1, p["res2_mult_a"], p["res2_mult_b"],
                                       p["res2_shift"]))
    return np.stack(out)


@pytest.mark.parametrize("variant", ["baseline", "wide"])
@pytest.mark.parametrize("win", [(0, 0), (4, 4)])
def test_block_equals_operator_chain(orc, variant, win):
    rng = np.random.Generator(np.random.PCG64(5))
    p = synth.block_params(rng, 64, 2, 32, 256, variant)
    x = rng.integers(-127, 128, (2, 64, 64)).astype(np.int8)
    y = orc.block_forward(p, x, 8, 8, *win)
    assert np.array_equal(y, chain_block(orc, p, x, 8, 8, *win))
    # batch independence
    assert np.array_equal(orc.block_forward(p, x[1:], 8, 8, *win), y[1:])


def test_saturation_per_requant_point(orc):
    """Saturation at every requantization point of the 256-token block: the
    baseline distributions (shifts 30-38) saturate most linear outputs, the
    wide variant (shifts 38-43) keeps each point mostly inside int8, so the
    wide parity runs exercise the rounding of every requantization."""
    wl = synth.WORKLOADS["block_t256_d192"]
    frac = {}
    for variant in ("baseline", "wide"):
        blocks, x = synth.encoder_inputs(wl, 101, variant)
        p, xb = blocks[0], x[0]
        sat = lambda t: float(np.mean(np.abs(t.astype(np.int64)) == 127))
        h = orc.int_layernorm(xb, p["ln1_beta"], p["ln1_mult"], p["ln1_shift"], p["ln_iters"])
        qkv = orc.linear(h, p["w_qkv"], p["b_qkv"], p["qkv_mult"], p["qkv_shift"])
        a = orc.attention(qkv, 16, 16, 0, 0, p["heads"], p["head_dim"], p["score_mult"],
                          p["score_shift"], p["smax_I0"], p["pv_mult"], p["pv_shift"])
        pr = orc.linear(a, p["w_proj"], p["b_proj"], p["proj_mult"], p["proj_shift"])
        x1 = orc.residual_tensor(pr, xb, p["res1_mult_a"], p["res1_mult_b"], p["res1_shift"])
        h2 = orc.int_layernorm(x1, p["ln2_beta"], p["ln2_mult"], p["ln2_shift"], p["ln_iters"])
        f1 = orc.linear(h2, p["w_fc1"], p["b_fc1"], p["fc1_mult"], p["fc1_shift"])
        g = orc.sdshiftgelu_tensor(f1, p["gelu_I0"], p["gelu_mult"], p["gelu_shift"])
        f2 = orc.linear(g, p["w_fc2"], p["b_fc2"], p["fc2_mult"], p["fc2_shift"])
        frac[variant] = {"LN1": sat(h), "QKV": sat(qkv), "attention": sat(a),
                         "projection": sat(pr), "LN2": sat(h2), "fc1": sat(f1), "GELU": sat(g),
                         "fc2": sat(f2)}
    for point in ("QKV", "projection", "fc1", "fc2"):
        assert frac["baseline"][point] > 0.5
    assert all(v < 0.25 for v in frac["wide"].values()), frac["wide"]


def test_block_wide_variant_is_not_saturated(orc):
    """The wide parity variant keeps most requantized values inside int8, so
    block parity exercises the rounding paths, not only saturation."""
    wl = synth.WORKLOADS["block_t256_d192"]
    blocks, x = synth.encoder_inputs(wl, 101, "wide")
    y = orc.block_forward(blocks[0], x, 16, 16, 0, 0)
    assert np.mean(np.abs(y) == 127) < 0.5
    assert len(np.unique(y)) > 100


# ------------------------------------------------------------------ deformable sampling
def _grid_sample(value_map, X, Y, W, H, mode):
    """torch grid_sample on the CPU; X, Y are Q8 'loc * size' coordinates."""
    gx = 2.0 * (X / 256.0) / W - 1.0
    gy = 2.0 * (Y / 256.0) / H - 1.0
    grid = torch.tensor(np.stack([gx, gy], -1), dtype=torch.float64).view(1, -1, 1, 2)
    inp = torch.tensor(value_map, dtype=torch.float64)[None]
    out = torch.nn.functional.grid_sample(inp, grid, mode=mode, padding_mode="zeros",
                                          align_corners=False)
    return out[0, :, :, 0].numpy()  # [C, n]


def test_nearest_index_matches_grid_sample(orc):
    rng = np.random.default_rng(6)
    for H, W in ((20, 20), (40, 40), (7, 13)):
        n = 3000
        rx = rng.integers(0, 65536, n)
        ry = rng.integers(0, 65536, n)
        ox = rng.integers(-2048, 2049, n)
        oy = rng.integers(-2048, 2049, n)
        X = (rx * W) // 256 + ox
        Y = (ry * H) // 256 + oy
        keep = (X % 256 != 0) & (Y % 256 != 0)  # exact half-pixel ties excluded
        idx_map = (np.arange(H * W, dtype=np.float64) + 1).reshape(1, H, W)
        gs = _grid_sample(idx_map, X, Y, W, H, "nearest")[0]
        for i in np.nonzero(keep)[0]:
            got = orc.deform_nearest_index(rx[i], ry[i], ox[i], oy[i], H, W)
            assert got + 1 == int(gs[i]), (H, W, i)


def _deform_inputs(seed, B=2, Q=5):
    wl = synth.DEFORM_WORKLOADS["deform_q300_d256_b8"]
    small = synth.DeformWorkload("small", B, Q, 64, 4, 16, ((10, 10), (5, 7), (3, 3)), 2)
    return synth.deform_inputs(small, seed), small


@pytest.mark.parametrize("mode,gs_mode", [(0, "nearest"), (1, "bilinear")])
def test_deform_attn_against_grid_sample(orc, mode, gs_mode):
    d, wl = _deform_inputs(7)
    offs = d["offsets"].copy()
    out = orc.deform_attn(d["value"], d["level_hw"], d["level_start"], d["ref"], offs,
                          d["logits"], d["I0"], d["out_mult"], d["out_shift"], mode)
    B, Q, H, L, P, _ = offs.shape
    Dh = d["value"].shape[-1]
    for b in range(B):
        for h in range(H):
            acc = np.zeros((Q, Dh))
            Pw = np.stack([orc.shiftmax_row(d["logits"][b, q, h], d["I0"])[0]
                           for q in range(Q)])
            for l in range(L):
                Hl, Wl = d["level_hw"][l]
                s0 = d["level_start"][l]
                vmap = d["value"][b, s0:s0 + Hl * Wl, h, :].reshape(Hl, Wl, Dh)
                vmap = vmap.transpose(2, 0, 1).astype(np.float64)
                for pt in range(P):
                    X = (d["ref"][b, :, 0].astype(np.int64) * Wl) // 256 + offs[b, :, h, l, pt, 0]
                    Y = (d["ref"][b, :, 1].astype(np.int64) * Hl) // 256 + offs[b, :, h, l, pt, 1]
                    gs = _grid_sample(vmap, X, Y, Wl, Hl, gs_mode)  # [Dh, Q]
                    acc += Pw[:, l * P + pt][:, None] * gs.T
            m, s = d["out_mult"], d["out_shift"]
            ref = np.clip(np.floor(acc * m / 2.0 ** s + 0.5), -127, 127)
            got = out[b, :, h * Dh:(h + 1) * Dh].astype(np.float64)
            tie = np.abs(acc * m / 2.0 ** s + 0.5 - np.round(acc * m / 2.0 ** s + 0.5)) < 1e-6
            if mode == 0:
                # nearest: exact unless a sample sits on a half-pixel tie
                assert np.mean(got == ref) > 0.98
            else:
                assert np.all((np.abs(got - ref) <= 1) | tie)
                assert np.mean(got == ref) > 0.98


def test_deform_zero_offsets_at_pixel_centres(orc):
    """Reference points on pixel centres with zero offsets sample that pixel:
    the output is the requantized sum of the Shiftmax weights times it."""
    d, wl = _deform_inputs(8, B=1, Q=3)
    L = len(wl.levels)
    offs = np.zeros_like(d["offsets"])
    # ref = (i + 0.5) / W in Q16 for a pixel i that exists on every level
    ref = np.zeros_like(d["ref"])
    for q in range(3):
        ref[0, q] = [int((q + 0.5) / 3 * 65536), int((2 - q + 0.5) / 3 * 65536)]
    out = orc.deform_attn(d["value"], d["level_hw"], d["level_start"], ref, offs,
                          d["logits"], d["I0"], 1 << 30, 30, 0)
    Dh = d["value"].shape[-1]
    for q in range(3):
        for h in range(wl.heads):
            Pw = orc.shiftmax_row(d["logits"][0, q, h], d["I0"])[0]
            acc = np.zeros(Dh, np.int64)
            for l in range(L):
                Hl, Wl = d["level_hw"][l]
                ix = (int(ref[0, q, 0]) * Wl) >> 16
                iy = (int(ref[0, q, 1]) * Hl) >> 16
                v = d["value"][0, d["level_start"][l] + iy * Wl + ix, h].astype(np.int64)
                acc += int(Pw[l * wl.points:(l + 1) * wl.points].sum()) * v
            assert np.array_equal(out[0, q, h * Dh:(h + 1) * Dh],
                                  np.clip(acc, -127, 127).astype(np.int8))


def test_deform_samples_outside_the_map_contribute_nothing(orc):
    d, _ = _deform_inputs(9)
    offs = np.full_like(d["offsets"], -30000)
    out = orc.deform_attn(d["value"], d["level_hw"], d["level_start"], d["ref"], offs,
                          d["logits"], d["I0"], d["out_mult"], d["out_shift"], 0)
    assert np.all(out == 0)
