"""GPU parity of the affine activation path (Eq. affine_q, Eq. uniform_q, Eq.
integer_accumulation with activation zero points): hatq_fwht_quant_act_affine,
hatq_weight_tapsums and hatq_conv_int8_affine against the oracle.

* Codes, scale and zero point bit-exact where both sides see identical fp32
  transform outputs (no transform, or dyadic integer inputs whose butterfly
  is exact); otherwise the scale within 1 ulp and codes under the INT8 rule.
* Centered INT32 accumulators bit-exact on every conv geometry (the oracle sums
  x - z over the pixels inside the image; the GPU subtracts z times the weight
  sum of the inside taps), transposed included.
* Dequantized fp32 outputs within 1e-6 of the range.
"""
import numpy as np
import pytest
import torch

from gpu_util import CODE_FLIP_FRACTION, assert_range_rel, assert_scale_ulp, dev, host, set_codes
from paper_2608_01653_amd import hatq, synth
from test_gpu_parity import CONV, CONV_IDS, _layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    hatq.load()
    torch.cuda.init()


def assert_codes(q_gpu, q_ref, exact=False, what="codes"):
    """The INT8 rule of the symmetric codes on the affine grid [-128, 127]."""
    d = np.abs(q_gpu.astype(np.int32) - q_ref.astype(np.int32))
    if exact:
        assert d.max() == 0, f"{what}: {np.count_nonzero(d)} of {d.size} differ (max {d.max()})"
    else:
        frac = np.count_nonzero(d) / d.size
        assert d.max() <= 1 and frac <= CODE_FLIP_FRACTION, f"{what}: max diff {d.max()}, fraction {frac:.3g}"


def _shifted(rng, shape):
    x = synth.heavy_tailed_activations(rng, shape)
    x[0] += np.float32(1.0) * np.abs(x[0]).mean()             # a positive mean on sample 0
    x[-1] = np.abs(x[-1])                                     # one-signed last sample: z at the grid's end
    return x


@pytest.mark.parametrize("shape", [(3, 31, 29, 64), (2, 17, 13, 3 * 4), (3, 64, 64, 192)])
def test_affine_quant_original_domain_bit_exact(orc, shape):
    rng = np.random.default_rng(sum(shape))
    x = _shifted(rng, shape)
    q_ref, s_ref, z_ref = orc.quantize_affine(x)
    q, s, z = hatq.hatq_fwht_quant_act_affine(dev(x), 1)
    assert np.array_equal(host(s), s_ref) and np.array_equal(host(z), z_ref)
    assert_codes(host(q), q_ref, exact=True, what="affine codes b=1")
    assert int(host(z)[-1]) == -128


@pytest.mark.parametrize("b", [2, 8, 64, 128])
def test_affine_quant_exact_transform_bit_exact(orc, b):
    rng = np.random.default_rng(200 + b)
    C = 256 if b == 128 else 192
    x = synth.dyadic_integers(rng, (3, 7, 9, C))
    x[1] += np.float32(3.0)
    S = orc.activation_transform(x, b)
    q_ref, s_ref, z_ref = orc.quantize_affine(S)
    q, s, z = hatq.hatq_fwht_quant_act_affine(dev(x), b)
    assert np.array_equal(host(s), s_ref) and np.array_equal(host(z), z_ref)
    assert_codes(host(q), q_ref, exact=True, what=f"affine codes b={b}")


def test_affine_quant_heavy_tailed(orc):
    rng = np.random.default_rng(210)
    x = _shifted(rng, (3, 33, 17, 192))
    S = orc.activation_transform(x, 64)
    q_ref, s_ref, z_ref = orc.quantize_affine(S)
    q, s, z = hatq.hatq_fwht_quant_act_affine(dev(x), 64)
    assert_scale_ulp(host(s), s_ref)
    assert np.abs(host(z).astype(np.int64) - z_ref).max() <= 1
    assert_codes(host(q), q_ref)


def test_affine_quant_zero_input():
    x = torch.zeros((2, 4, 4, 64), device="cuda")
    q, s, z = hatq.hatq_fwht_quant_act_affine(x, 64)
    assert torch.all(s == 1) and not torch.any(z) and not torch.any(q)


def _tapsums_ref(wq_ohwi):
    cout_p, k, _, cin_p = wq_ohwi.shape
    per = wq_ohwi.astype(np.int64).sum(axis=3).reshape(cout_p, k * k).T      # [k*k][cout_p]
    return np.concatenate([per, per.sum(axis=0, keepdims=True)]).astype(np.int32)


@pytest.mark.parametrize("c", CONV, ids=CONV_IDS)
def test_affine_conv_int32_bit_exact(orc, c):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 211)
    xq = synth.int8_codes(rng, (n, h, w, ref.cin_p))
    wq = synth.int8_codes(rng, ref.wq.shape)
    set_codes(layer, wq)
    zx = rng.integers(-128, 128, n).astype(np.int32)
    zx[0] = -128
    tapsum = hatq.hatq_weight_tapsums(layer)
    assert np.array_equal(host(tapsum).reshape(k * k + 1, -1), _tapsums_ref(wq))
    acc_ref = orc.conv_int8(xq, wq, stride=s, pad=p, transposed=tr, out_pad=op, zx=zx)
    acc = hatq.hatq_conv_int8_affine(layer, dev(xq), torch.ones(n, device="cuda"), dev(zx), tapsum,
                                     hatq.HATQ_OUT_I32)
    assert np.array_equal(host(acc), acc_ref)


@pytest.mark.parametrize("ci", [1, 2, 4, 5, 7, 12, 15], ids=[CONV_IDS[i] for i in (1, 2, 4, 5, 7, 12, 15)])
def test_affine_layer_f32(orc, ci):
    """The whole affine layer: the oracle's codes, scale and zero point feed the
    GPU convolution; the fp32 output matches the oracle's epilogue of its
    centered accumulators."""
    c = CONV[ci]
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 212)
    x = _shifted(rng, (n, h, w, cin))
    S = orc.activation_transform(x, hb if form == "DH" else 1)
    xq, sx, zx = orc.quantize_affine(S)
    if xq.shape[-1] < ref.cin_p:
        xq = np.concatenate([xq, np.zeros(xq.shape[:-1] + (ref.cin_p - xq.shape[-1],), np.int8)], axis=-1)
    acc_ref = orc.conv_int8(xq, ref.wq, stride=s, pad=p, transposed=tr, out_pad=op, zx=zx)
    y_ref = orc.epilogue(acc_ref, sx, ref)
    tapsum = hatq.hatq_weight_tapsums(layer)
    y = hatq.hatq_conv_int8_affine(layer, dev(xq), dev(sx), dev(zx), tapsum, hatq.HATQ_OUT_F32)
    assert_range_rel(host(y), y_ref, what="affine layer y")
