"""Pins of the oracle's deformable sampling with reference boxes (the
decoder's reference boxes, Sec. 3.1.2, with the sampling offsets taken
relative to the box as in the deformable decoder the paper builds on; the
paper gives no formula, so the location rule is a reading):

    location = c + (off / 2^8) / P * size / 2     (fractions of the map)

* nearest indices against torch's grid_sample on the CPU (half-pixel
  convention, zero padding), computed from the real-valued location;
* the whole sampler against grid_sample (nearest and bilinear) at box
  references;
* zero offsets sample the box centre, i.e. the point form at (cx, cy);
* a box of 2P pixels turns box units into pixels: the point form exactly;
* only the product off * size matters (doubling the size and halving the
  offsets changes nothing), and width and height act on x and y separately.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_24981_amd import synth


def _grid_sample(value_map, Xr, Yr, W, H, mode):
    """torch grid_sample on the CPU at real-valued Q8 pixel coordinates."""
    gx = 2.0 * (Xr / 256.0) / W - 1.0
    gy = 2.0 * (Yr / 256.0) / H - 1.0
    grid = torch.tensor(np.stack([gx, gy], -1), dtype=torch.float64).view(1, -1, 1, 2)
    inp = torch.tensor(value_map, dtype=torch.float64)[None]
    out = torch.nn.functional.grid_sample(inp, grid, mode=mode, padding_mode="zeros",
                                          align_corners=False)
    return out[0, :, :, 0].numpy()


def _box_location(c, size, off, P, W):
    """Real-valued Q8 pixel coordinate of a box-relative sample."""
    loc = c / 65536.0 + (off / 256.0) / P * (size / 65536.0) / 2.0
    return loc * W * 256.0


def test_box_nearest_index_matches_grid_sample():
    rng = np.random.default_rng(11)
    for H, W, P in ((20, 20, 4), (40, 40, 4), (7, 13, 3), (80, 80, 1)):
        n = 3000
        cx, cy = rng.integers(0, 65536, n), rng.integers(0, 65536, n)
        w, h = rng.integers(1 << 12, 1 << 16, n), rng.integers(1 << 12, 1 << 16, n)
        ox, oy = rng.integers(-2048, 2049, n), rng.integers(-2048, 2049, n)
        Xr = _box_location(cx, w, ox, P, W)
        Yr = _box_location(cy, h, oy, P, H)
        # exact pixel-boundary ties excluded (round-half-even in grid_sample)
        keep = (np.abs(Xr / 256 - np.round(Xr / 256)) > 1e-9) & \
               (np.abs(Yr / 256 - np.round(Yr / 256)) > 1e-9)
        idx_map = (np.arange(H * W, dtype=np.float64) + 1).reshape(1, H, W)
        gs = _grid_sample(idx_map, Xr, Yr, W, H, "nearest")[0]
        for i in np.nonzero(keep)[0]:
            got = oracle.deform_box_nearest_index(cx[i], cy[i], w[i], h[i], ox[i], oy[i],
                                                  H, W, P)
            assert got + 1 == int(gs[i]), (H, W, P, i)


def _small(seed, B=2, Q=5, levels=((10, 10), (5, 7), (3, 3)), P=2):
    wl = synth.DeformWorkload("small", B, Q, 64, 4, 16, levels, P)
    return synth.deform_inputs(wl, seed, boxes=True), wl


@pytest.mark.parametrize("mode,gs_mode", [(0, "nearest"), (1, "bilinear")])
def test_box_sampler_against_grid_sample(mode, gs_mode):
    d, wl = _small(21)
    offs = d["offsets"]
    out = oracle.deform_attn(d["value"], d["level_hw"], d["level_start"], d["ref"], offs,
                             d["logits"], d["I0"], d["out_mult"], d["out_shift"], mode)
    B, Q, H, L, P, _ = offs.shape
    Dh = d["value"].shape[-1]
    ref = d["ref"].astype(np.float64)
    agree = total = 0
    for b in range(B):
        for h in range(H):
            acc = np.zeros((Q, Dh))
            Pw = np.stack([oracle.shiftmax_row(d["logits"][b, q, h], d["I0"])[0]
                           for q in range(Q)])
            for l in range(L):
                Hl, Wl = d["level_hw"][l]
                s0 = d["level_start"][l]
                vmap = d["value"][b, s0:s0 + Hl * Wl, h, :].reshape(Hl, Wl, Dh)
                vmap = vmap.transpose(2, 0, 1).astype(np.float64)
                for pt in range(P):
                    Xr = _box_location(ref[b, :, 0], ref[b, :, 2], offs[b, :, h, l, pt, 0], P, Wl)
                    Yr = _box_location(ref[b, :, 1], ref[b, :, 3], offs[b, :, h, l, pt, 1], P, Hl)
                    if mode == 1:  # the oracle floors the location to Q8 first
                        Xr, Yr = np.floor(Xr), np.floor(Yr)
                    gs = _grid_sample(vmap, Xr, Yr, Wl, Hl, gs_mode)
                    acc += Pw[:, l * P + pt][:, None] * gs.T
            m, s = d["out_mult"], d["out_shift"]
            want = np.clip(np.floor(acc * m / 2.0 ** s + 0.5), -127, 127)
            got = out[b, :, h * Dh:(h + 1) * Dh].astype(np.float64)
            assert np.all(np.abs(got - want) <= 1)
            agree += np.sum(got == want)
            total += got.size
    assert agree / total > 0.98


@pytest.mark.parametrize("mode", [0, 1])
def test_zero_offsets_sample_the_box_centre(mode):
    """With zero offsets the box size plays no part: the point form at the
    box centre."""
    d, _ = _small(22)
    zero = np.zeros_like(d["offsets"])
    args = (d["logits"], d["I0"], d["out_mult"], d["out_shift"], mode)
    got = oracle.deform_attn(d["value"], d["level_hw"], d["level_start"], d["ref"], zero, *args)
    pts = np.ascontiguousarray(d["ref"][..., :2])
    assert np.array_equal(got, oracle.deform_attn(d["value"], d["level_hw"],
                                                  d["level_start"], pts, zero, *args))


@pytest.mark.parametrize("mode", [0, 1])
def test_box_of_2p_pixels_is_the_point_form(mode):
    """On a 64 x 32 map with P = 4, a box of w = 2^17 P / 64 and
    h = 2^17 P / 32 (2P pixels each way) makes one box unit one pixel, so
    every offset lands where the point form puts it."""
    d, wl = _small(23, levels=((32, 64),), P=4)
    B, Q = d["ref"].shape[:2]
    ref = d["ref"].copy()
    ref[..., 2] = (1 << 17) * 4 // 64
    ref[..., 3] = (1 << 17) * 4 // 32
    args = (d["offsets"], d["logits"], d["I0"], d["out_mult"], d["out_shift"], mode)
    got = oracle.deform_attn(d["value"], d["level_hw"], d["level_start"], ref, *args)
    pts = np.ascontiguousarray(ref[..., :2])
    assert np.array_equal(got, oracle.deform_attn(d["value"], d["level_hw"],
                                                  d["level_start"], pts, *args))
    # and the sampled pixels are not all the same one: the offsets matter
    moved = oracle.deform_attn(d["value"], d["level_hw"], d["level_start"], pts,
                               np.zeros_like(d["offsets"]), *args[1:])
    assert not np.array_equal(got, moved)


def test_only_offset_times_size_matters():
    """Doubling w (resp. h) and halving the x (resp. y) offsets leaves every
    location unchanged; changing w alone moves only x."""
    d, _ = _small(24)
    offs = (d["offsets"] // 2) * 2  # even offsets
    args = (d["logits"], d["I0"], d["out_mult"], d["out_shift"], 0)
    ref2 = d["ref"].copy()
    ref2[..., 2] //= 2
    ref2[..., 2] *= 2   # even widths
    ref2[..., 3] //= 2
    ref2[..., 3] *= 2
    even = oracle.deform_attn(d["value"], d["level_hw"], d["level_start"], ref2, offs, *args)
    ref3 = ref2.copy()
    ref3[..., 2:] //= 2
    offs3 = offs * 2
    assert np.array_equal(even, oracle.deform_attn(d["value"], d["level_hw"],
                                                   d["level_start"], ref3, offs3, *args))
    # the index rule itself: x depends on (w, off_x) only, y on (h, off_y) only
    for cx, cy, w, h, ox, oy in ((30000, 40000, 5000, 9000, 300, -700),
                                 (100, 65000, 20000, 4096, -2048, 2048)):
        a = oracle.deform_box_nearest_index(cx, cy, w, h, ox, oy, 40, 40, 4)
        b = oracle.deform_box_nearest_index(cx, cy, w, h * 2, ox, oy // 2, 40, 40, 4)
        c = oracle.deform_box_nearest_index(cx, cy, w * 2, h, ox // 2, oy, 40, 40, 4)
        assert a == b == c
