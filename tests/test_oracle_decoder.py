"""The oracle's decoder layer against the chain of its separately pinned
operators (linear layers, attention, residual adds, I-LayerNorm, deformable
sampling, SD-ShiftGELU), wired in the order the layer's reading states:
post-norm self-attention over the queries, deformable cross-attention with
int8 offsets in 1/16 pixel widened to Q8, FFN."""
import numpy as np
import pytest

import oracle
from paper_2607_24981_amd import synth


def chain(p, tgt, memory, ref, hw, start):
    B, Q, D = tgt.shape
    H, L, P = p["heads"], p["levels"], p["points"]
    lin = lambda x, stem: oracle.linear(x.reshape(-1, x.shape[-1]), p["w_" + stem],
                                        p["b_" + stem], p[stem + "_mult"], p[stem + "_shift"])
    ln = lambda x, stem: oracle.int_layernorm(x, p[stem + "_beta"], p[stem + "_mult"],
                                              p[stem + "_shift"], p["ln_iters"])
    res = lambda a, b, i: oracle.residual_tensor(a, b, p[f"res{i}_mult_a"],
                                                 p[f"res{i}_mult_b"], p[f"res{i}_shift"])
    att = np.stack([oracle.attention(lin(tgt[b], "qkv"), 1, Q, 0, 0, H, D // H,
                                     p["score_mult"], p["score_shift"], p["smax_I0"],
                                     p["pv_mult"], p["pv_shift"], s_d=p["smax_s_d"])
                    for b in range(B)]).reshape(B * Q, D)
    t1 = ln(res(lin(att, "o"), tgt.reshape(B * Q, D), 1), "ln1")
    v = lin(memory, "val").reshape(B, -1, H, D // H)
    off = (lin(t1, "off").astype(np.int16) * 16).reshape(B, Q, H, L, P, 2)
    lg = lin(t1, "attw").reshape(B, Q, H, L * P)
    smp = oracle.deform_attn(v, hw, start, ref, off, lg, p["da_I0"], p["da_out_mult"],
                             p["da_out_shift"], p["da_mode"], s_d=p["da_s_d"])
    t2 = ln(res(lin(smp, "co"), t1, 2), "ln2")
    f1 = lin(t2, "fc1")
    g = oracle.sdshiftgelu_tensor(f1, p["gelu_I0"], p["gelu_mult"], p["gelu_shift"])
    y = ln(res(lin(g, "fc2"), t2, 3), "ln3")
    return y.reshape(B, Q, D)


@pytest.mark.parametrize("boxes", [False, True])
@pytest.mark.parametrize("mode", [0, 1])
def test_decoder_equals_operator_chain(mode, boxes):
    """Point references and reference boxes (the sampler's box form)."""
    wl = synth.DecoderWorkload("small", 2, 37, 64, 2, 128, ((9, 13), (4, 6), (2, 3)), 3)
    p, tgt, mem, ref, hw, start = synth.decoder_inputs(wl, 11 + mode, mode=mode, boxes=boxes)
    y = oracle.decoder_forward(p, tgt, mem, ref, hw, start)
    assert np.array_equal(y, chain(p, tgt, mem, ref, hw, start))
    assert np.std(y.astype(np.float64)) > 5


def test_decoder_layernorm_iterations_are_used():
    """The decoder's LayerNorms run the Newton count they are given (20 in
    the paper's decoder): with 1 step the output changes."""
    wl = synth.DecoderWorkload("small", 1, 16, 64, 2, 128, ((8, 8),), 2)
    p, tgt, mem, ref, hw, start = synth.decoder_inputs(wl, 3)
    y20 = oracle.decoder_forward(p, tgt, mem, ref, hw, start)
    y1 = oracle.decoder_forward(dict(p, ln_iters=1), tgt, mem, ref, hw, start)
    assert not np.array_equal(y20, y1)
