"""Out-of-bounds writes and the non-finite input contract, through the C ABI.

* Canaries: every entry point writes its outputs into buffers with guard bytes
  on both sides, on geometries with ragged tiles (sizes that are not multiples
  of any tile, odd batch sizes, channel counts that leave partial column
  tiles); no guard byte may change.
* Non-finite inputs (NaN, +-Inf) are outside the operator's contract: the codes
  and scale of a sample that holds one are unspecified, but the kernels
  complete, every other sample's codes and scale are those it gets alone (one
  scale per sample), and nothing outside the outputs is written.
"""
import numpy as np
import pytest
import torch

from gpu_util import Guarded, dev, host
from paper_2608_01653_amd import hatq, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    hatq.load()
    torch.cuda.init()


@pytest.mark.parametrize("shape,b", [((3, 13, 11, 192), 64), ((1, 7, 5, 128), 128), ((5, 9, 7, 3), 1),
                                     ((2, 5, 3, 2), 1), ((3, 6, 7, 192), 192)])
def test_act_quant_guards(shape, b):
    rng = np.random.default_rng(3000 + b)
    x = dev(synth.heavy_tailed_activations(rng, shape))
    q = Guarded(shape, torch.int8)
    s = Guarded((shape[0],), torch.float32)
    hatq.hatq_fwht_quant_act(x, b, xq=q.view, scale=s.view)
    q.check("codes")
    s.check("scale")
    q_ref, s_ref = hatq.hatq_fwht_quant_act(x, b)
    assert torch.equal(q.view, q_ref) and torch.equal(s.view, s_ref)


# (n, h, w, cin, cout, k, stride, pad, transposed, out_pad, form, hblock)
CONV = [(3, 13, 17, 192, 192, 5, 2, 2, False, 0, "DH", 64),
        (1, 21, 9, 192, 320, 5, 2, 2, False, 0, "WH", 64),
        (2, 11, 19, 3, 192, 5, 2, 2, False, 0, "WH", 64),
        (2, 7, 5, 192, 192, 5, 2, 2, True, 1, "DH", 64),
        (1, 9, 11, 128, 128, 1, 1, 0, False, 0, "DH", 128),
        (2, 5, 13, 64, 192, 3, 1, 1, False, 0, "WH", 64)]
IDS = [f"{c[10]}{c[3]}-{c[4]}k{c[5]}s{c[6]}{'t' if c[8] else ''}" for c in CONV]


def _layer(c, seed):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng = np.random.default_rng(seed)
    wt, b = synth.layer_params(rng, cin, cout, k, tr)
    layer = hatq.hatq_prepare_weights(hatq.desc(cin, cout, k, s, p, hb, tr, op), form, dev(wt), dev(b))
    xq = dev(synth.int8_codes(rng, (n, h, w, layer.w.cin_pad)))
    sx = dev(rng.uniform(1e-3, 1e-2, n).astype(np.float32))
    return layer, xq, sx


@pytest.mark.parametrize("c", CONV, ids=IDS)
def test_conv_guards(c):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    layer, xq, sx = _layer(c, 3100)
    ho, wo = hatq.hatq_conv_out_hw(layer.w.d, h, w)
    cp = layer.w.cout_pad
    # I32 and F32 outputs, with and without the next operand's absmax
    g32 = Guarded((n, ho, wo, cp), torch.int32)
    hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_I32, y=g32.view)
    g32.check("I32 output")
    gf = Guarded((n, ho, wo, cout), torch.float32)
    ga = Guarded((n,), torch.float32)
    hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32, next_hblock=64, next_absmax=ga.view, y=gf.view)
    gf.check("F32 output")
    ga.check("next absmax")
    y_plain = hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32)
    assert torch.equal(gf.view, y_plain)
    # the requantizing epilogue (dynamic scale) and the I8 mode of hatq_conv_int8 (static)
    gq = Guarded((n, ho, wo, cout), torch.int8)
    gs = Guarded((n,), torch.float32)
    hatq.hatq_conv_int8_requant(layer, xq, sx, 64, next_absmax=ga.view, next_scale=gs.view, yq=gq.view)
    gq.check("requantized codes")
    gs.check("next scale")
    g8 = Guarded((n, ho, wo, cout), torch.int8)
    hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_I8, next_hblock=64, out_scale=gs.view, y=g8.view)
    g8.check("I8 output")
    assert torch.equal(g8.view, gq.view)
    # the integer transition
    s_y = float(host(gs.view).max())
    table, _ = hatq.hatq_int_transition_params(layer, float(host(sx).max()), s_y, 64)
    gi = Guarded((n, ho, wo, cout), torch.int8)
    hatq.hatq_conv_int8_int_transition(layer, xq, 64, table, yq=gi.view)
    gi.check("integer transition codes")
    # affine codes with zero point 0: the symmetric result
    zx = torch.zeros(n, dtype=torch.int32, device="cuda")
    ts = hatq.hatq_weight_tapsums(layer)
    gaf = Guarded((n, ho, wo, cout), torch.float32)
    hatq.hatq_conv_int8_affine(layer, xq, sx, zx, ts, hatq.HATQ_OUT_F32, y=gaf.view)
    gaf.check("affine F32 output")
    assert torch.equal(gaf.view, y_plain)


def test_layer_forward_and_profiling_guards():
    rng = np.random.default_rng(3200)
    x = dev(synth.heavy_tailed_activations(rng, (3, 13, 17, 192)))
    wt, b = synth.layer_params(rng, 192, 192, 5)
    layer = hatq.hatq_prepare_weights(hatq.desc(192, 192, 5, 2, 2, 64), "DH", dev(wt), dev(b))
    gy = Guarded((3, 7, 9, 192), torch.float32)
    hatq.hatq_layer_forward(layer, "DH", x, y=gy.view)
    gy.check("layer output")
    gam = Guarded((6,), torch.float32)
    gfl = Guarded((3,), torch.int32)
    hatq.hatq_range_expansion(x, 64, amax=gam.view, flags=gfl.view)
    gam.check("range maxima")
    gfl.check("range flags")
    q = Guarded((3, 13, 17, 192), torch.int8)
    s = Guarded((3,), torch.float32)
    z = Guarded((3,), torch.int32)
    hatq.hatq_fwht_quant_act_affine(x, 64, xq=q.view, scale=s.view, zero=z.view)
    q.check("affine codes")
    s.check("affine scale")
    z.check("affine zero point")


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), -float("inf")])
@pytest.mark.parametrize("b", [64, 1])
def test_non_finite_input_contract(bad, b):
    rng = np.random.default_rng(3300)
    x_np = synth.heavy_tailed_activations(rng, (3, 9, 11, 192))
    x_bad = x_np.copy()
    x_bad[1, 4, 5, 17] = bad                       # sample 1 holds one non-finite value
    q = Guarded(x_np.shape, torch.int8)
    s = Guarded((3,), torch.float32)
    hatq.hatq_fwht_quant_act(dev(x_bad), b, xq=q.view, scale=s.view)
    q.check("codes")
    s.check("scale")
    for k in (0, 2):                               # the other samples: as if alone
        q1, s1 = hatq.hatq_fwht_quant_act(dev(np.ascontiguousarray(x_np[k:k + 1])), b)
        assert torch.equal(q.view[k:k + 1], q1) and torch.equal(s.view[k:k + 1], s1)
    # a layer whose input holds it: completes, and other samples' outputs are unchanged
    wt, bias = synth.layer_params(rng, 192, 192, 5)
    layer = hatq.hatq_prepare_weights(hatq.desc(192, 192, 5, 2, 2, 64), "DH", dev(wt), dev(bias))
    y_bad = hatq.hatq_layer_forward(layer, "DH", dev(x_bad))
    y_ok = hatq.hatq_layer_forward(layer, "DH", dev(x_np))
    torch.cuda.synchronize()
    assert torch.equal(y_bad[0], y_ok[0]) and torch.equal(y_bad[2], y_ok[2])
