"""GPU parity of the Kronecker transform orders 192 = P_12 (x) H~_16 and
320 = P_20 (x) H~_16 (Eq. hadamard_order: m(192) = 192, m(320) = 320) for DH
layers: the activation transform and quantization, the weight preparation and
whole layers, against the oracle's dense construction of the same matrices.

* Dyadic integer inputs make every fp32 partial sum of the butterfly and of the
  Paley stage exact, so codes and scales are bit-exact, and a DH layer's output
  is bit-exact.
* Heavy-tailed inputs: the scale within 1 ulp and codes under the INT8 rule.
* Weight preparation is an fp64 sum in the same order on both sides: bit-exact.
"""
import numpy as np
import pytest
import torch

from gpu_util import assert_codes, assert_range_rel, assert_scale_ulp, dev, host, unpack_codes
from paper_2608_01653_amd import hatq, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    hatq.load()
    torch.cuda.init()


@pytest.mark.parametrize("m", [192, 320])
def test_act_quant_exact_transform_bit_exact(orc, m):
    rng = np.random.default_rng(300 + m)
    x = synth.dyadic_integers(rng, (3, 7, 9, 2 * m))
    S, q_ref, s_ref = orc.activation_operand(x, "DH", m)
    q, s = hatq.hatq_fwht_quant_act(dev(x), m)
    assert np.array_equal(host(s), s_ref)
    assert_codes(host(q), q_ref, exact=True, what=f"codes m={m}")


@pytest.mark.parametrize("m", [192, 320])
def test_act_quant_heavy_tailed(orc, m):
    rng = np.random.default_rng(310 + m)
    x = synth.heavy_tailed_activations(rng, (2, 33, 17, m))
    S, q_ref, s_ref = orc.activation_operand(x, "DH", m)
    q, s = hatq.hatq_fwht_quant_act(dev(x), m)
    assert_scale_ulp(host(s), s_ref)
    assert_codes(host(q), q_ref)
    # the fused-absmax entry (absmax given) reads once and gives the same codes
    A = torch.tensor(np.abs(S.reshape(2, -1)).max(axis=1), device="cuda")
    q2, s2 = hatq.hatq_fwht_quant_act(dev(x), m, absmax=A)
    assert np.array_equal(host(s2), s_ref)


LAYERS = [  # (n, h, w, cin, cout, k, stride, pad, transposed, out_pad, form, hblock)
    (2, 21, 19, 192, 192, 5, 2, 2, False, 0, "DH", 192),     # window kernel
    (1, 17, 23, 320, 192, 5, 2, 2, False, 0, "DH", 320),
    (1, 13, 11, 192, 128, 3, 1, 1, False, 0, "DH", 192),     # pipeline kernel
    (1, 6, 7, 192, 192, 5, 2, 2, True, 1, "DH", 192),        # transposed phases
]
IDS = [f"{c[3]}to{c[4]}-k{c[5]}s{c[6]}-m{c[11]}{'-T' if c[8] else ''}" for c in LAYERS]


def _layer(orc, c, seed):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng = np.random.default_rng(seed)
    wt, b = synth.layer_params(rng, cin, cout, k, tr)
    ref = orc.prepare_weights(wt, b, cin=cin, cout=cout, k=k, stride=s, pad=p, form=form, hblock=hb,
                              transposed=tr, out_pad=op)
    layer = hatq.hatq_prepare_weights(hatq.desc(cin, cout, k, s, p, hb, tr, op), form, dev(wt), dev(b))
    return rng, ref, layer


@pytest.mark.parametrize("c", LAYERS, ids=IDS)
def test_prepare_weights_bit_exact(orc, c):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, ref, layer = _layer(orc, c, 320)
    assert np.array_equal(unpack_codes(layer, k, ref.cin_p), ref.wq)
    assert np.array_equal(host(layer.w_scale()), ref.w_scale)
    assert np.array_equal(host(layer.bias()), ref.w_bias)


@pytest.mark.parametrize("c", LAYERS, ids=IDS)
def test_layer_forward_exact_inputs(orc, c):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, ref, layer = _layer(orc, c, 321)
    x = synth.dyadic_integers(rng, (n, h, w, cin))
    r = orc.layer_forward(x, ref)
    sc = torch.empty(n, device="cuda")
    y = host(hatq.hatq_layer_forward(layer, form, dev(x), act_scale=sc))
    assert np.array_equal(host(sc), r.sx)
    assert np.array_equal(y, r.y)


@pytest.mark.parametrize("c", LAYERS[:2], ids=IDS[:2])
def test_layer_forward_heavy_tailed(orc, c):
    """The oracle's codes and scale fed to the GPU convolution: fp32 output
    within 1e-6 of the range; the whole GPU layer within the code rule."""
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, ref, layer = _layer(orc, c, 322)
    x = synth.heavy_tailed_activations(rng, (n, h, w, cin))
    r = orc.layer_forward(x, ref)
    y = hatq.hatq_conv_int8(layer, dev(r.xq), dev(r.sx), hatq.HATQ_OUT_F32)
    assert_range_rel(host(y), r.y)


def test_unsupported_uses_are_rejected(orc):
    c = LAYERS[0]
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    _, ref, layer = _layer(orc, c, 323)
    xq = torch.zeros((n, h, w, cin), dtype=torch.int8, device="cuda")
    sx = torch.ones(n, device="cuda")
    with pytest.raises(hatq.HatqError):
        hatq.hatq_conv_int8_requant(layer, xq, sx, 64, next_scale=torch.ones(n, device="cuda"))
    with pytest.raises(hatq.HatqError):
        hatq.hatq_range_expansion(torch.zeros((1, 2, 2, 192), device="cuda"), 192)
    wh = hatq.hatq_prepare_weights(hatq.desc(64, 192, 3, 1, 1, 192), "WH",
                                   torch.ones(192, 64, 3, 3, device="cuda"), torch.zeros(192, device="cuda"))
    with pytest.raises(hatq.HatqError):      # the WH restore runs power-of-two blocks only
        hatq.hatq_conv_int8(wh, torch.zeros((1, 8, 8, 64), dtype=torch.int8, device="cuda"),
                            torch.ones(1, device="cuda"), hatq.HATQ_OUT_F32)
