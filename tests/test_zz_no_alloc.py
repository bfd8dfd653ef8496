"""The allocation-free block entry point (ilw_block_forward_noalloc): the
library's static device scratch in place of a caller workspace, checked
against ilw_block_forward with a workspace, bit for bit, on consecutive calls
of decreasing size (the scratch keeps the previous call's bytes), and against
the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_24981_amd import ilw, synth

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _poisoned_like(x):
    y = torch.empty_like(x)
    y.view(torch.uint8).fill_(0x5A)
    return y


def _case(seed, B, grid, win):
    g = np.random.Generator(np.random.PCG64(seed))
    p = synth.block_params(g, 192, 3, 64, 768, "wide")
    x = g.integers(-127, 128, (B, grid[0] * grid[1], 192)).astype(np.int8)
    return p, x


def _one(p, x, grid, win):
    print(f"[gpu] noalloc block B={x.shape[0]} grid={grid} win={win}", flush=True)
    blk = ilw.DeviceBlock(p)
    xd = ilw.to_device(x)
    want = ilw.ilw_block_forward(blk, xd, *grid, *win, y=_poisoned_like(xd))
    got = ilw.ilw_block_forward_noalloc(blk, xd, *grid, *win, y=_poisoned_like(xd))
    torch.cuda.synchronize()
    w, gt = want.cpu().numpy(), got.cpu().numpy()
    assert np.array_equal(gt, w), f"{np.count_nonzero(gt != w)} of {w.size} differ"
    return gt


def test_noalloc_matches_workspace_entry_twice():
    """Two calls in a row, the second on a smaller input (fewer images, a
    smaller grid, windowed attention), each against the workspace entry
    point; the first also against the oracle."""
    p, x = _case(11, 3, (16, 16), (0, 0))
    first = _one(p, x, (16, 16), (0, 0))
    ref = oracle.block_forward(p, x, 16, 16, 0, 0)
    assert np.array_equal(first, ref), "noalloc block differs from the oracle"
    p2, x2 = _case(12, 1, (8, 12), (4, 6))
    second = _one(p2, x2, (8, 12), (4, 6))
    ref2 = oracle.block_forward(p2, x2, 8, 12, 4, 6)
    assert np.array_equal(second, ref2), "second noalloc call differs from the oracle"


def test_noalloc_in_place():
    p, x = _case(13, 2, (10, 10), (5, 5))
    blk = ilw.DeviceBlock(p)
    want = ilw.ilw_block_forward(blk, ilw.to_device(x), 10, 10, 5, 5)
    t = ilw.to_device(x)
    ilw.ilw_block_forward_noalloc(blk, t, 10, 10, 5, 5, y=t)
    torch.cuda.synchronize()
    assert np.array_equal(t.cpu().numpy(), want.cpu().numpy())


def test_noalloc_rejects_oversize():
    """A block whose workspace need exceeds the static scratch is refused on
    the host with ILW_E_WORKSPACE, and the output is left untouched."""
    g = np.random.Generator(np.random.PCG64(14))
    p = synth.block_params(g, 384, 6, 64, 1536, "wide")
    blk = ilw.DeviceBlock(p)
    B = 8
    need = blk.workspace_bytes(B, 40, 40, 20, 20)
    assert need > ilw.NOALLOC_SCRATCH_BYTES
    xd = torch.zeros((B, 1600, 384), dtype=torch.int8, device="cuda")
    y = _poisoned_like(xd)
    with pytest.raises(ilw.IlwError, match="status -5"):
        ilw.ilw_block_forward_noalloc(blk, xd, 40, 40, 20, 20, y=y)
    torch.cuda.synchronize()
    assert bool((y.view(torch.uint8) == 0x5A).all())
