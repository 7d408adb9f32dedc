"""GPU parity of every stage of the HIP path against the CPU oracle, at sizes the
oracle finishes in seconds that still span several tiles and ragged tails:
activation transform + quantization, weight preparation, INT8 convolution
(INT32 accumulators), the DH/WH epilogues, the fused next-operand absmax and the
whole layer.  All calls go through the C ABI (libhatq.so)."""
import numpy as np
import pytest
import torch

from gpu_util import (assert_codes, assert_range_rel, assert_scale_ulp, dev, expected_pack, host,
                      set_codes, unpack_codes)
from paper_2608_01653_amd import hatq, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    hatq.load()
    torch.cuda.init()


# -------------------------------------------------------------------- a2-a4
@pytest.mark.parametrize("b", [1, 2, 4, 8, 16, 32, 64, 128])
def test_act_quant_exact_transform_bit_exact(orc, b):
    """Dyadic integer inputs: every fp32 butterfly partial sum is exact, so GPU
    and oracle see identical transform outputs and codes must match bit for bit."""
    rng = np.random.default_rng(100 + b)
    C = 256 if b == 128 else 192
    x = synth.dyadic_integers(rng, (3, 7, 9, C))
    S, q_ref, s_ref = orc.activation_operand(x, "DH", b)
    q, s = hatq.hatq_fwht_quant_act(dev(x), b)
    assert_codes(host(q), q_ref, exact=True)
    assert np.array_equal(host(s), s_ref)


@pytest.mark.parametrize("shape,b", [((1, 64, 64, 128), 128), ((2, 33, 17, 192), 64),
                                     ((1, 50, 40, 64), 64), ((3, 11, 13, 128), 32)])
def test_act_quant_heavy_tailed(orc, shape, b):
    rng = np.random.default_rng(7)
    x = synth.heavy_tailed_activations(rng, shape)
    S, q_ref, s_ref = orc.activation_operand(x, "DH", b)
    q, s = hatq.hatq_fwht_quant_act(dev(x), b)
    assert_scale_ulp(host(s), s_ref)
    assert_codes(host(q), q_ref)


@pytest.mark.parametrize("shape", [(1, 256, 256, 192), (2, 31, 29, 3), (2, 3, 5, 3), (1, 7, 7, 2)])
def test_act_quant_original_domain_bit_exact(orc, shape):
    """WH activations (b = 1): no transform, so codes are always bit-exact.
    (2,3,5,3) and (1,7,7,2) have h*w*c not a multiple of 4: elementwise path."""
    rng = np.random.default_rng(8)
    x = synth.heavy_tailed_activations(rng, shape)
    _, q_ref, s_ref = orc.activation_operand(x, "WH", 64)
    q, s = hatq.hatq_fwht_quant_act(dev(x), 1)
    assert np.array_equal(host(s), s_ref)
    assert_codes(host(q), q_ref, exact=True)


def test_act_quant_given_absmax(orc):
    """With the per-sample max |S| supplied (the fused path), the single-read
    kernel gives the oracle's codes; and it equals the two-pass result."""
    rng = np.random.default_rng(9)
    x = synth.dyadic_integers(rng, (2, 21, 19, 192))
    S, q_ref, s_ref = orc.activation_operand(x, "DH", 64)
    A = np.abs(S.reshape(2, -1)).max(1).astype(np.float32)
    q1, s1 = hatq.hatq_fwht_quant_act(dev(x), 64, absmax=dev(A))
    q2, s2 = hatq.hatq_fwht_quant_act(dev(x), 64)
    assert_codes(host(q1), q_ref, exact=True)
    assert np.array_equal(host(s1), s_ref)
    assert torch.equal(q1, q2) and torch.equal(s1, s2)


def test_act_quant_zero_and_ties(orc):
    z = np.zeros((2, 4, 4, 64), np.float32)
    q, s = hatq.hatq_fwht_quant_act(dev(z), 64)
    assert np.all(host(s) == 1.0) and not host(q).any()
    # s = 1 exactly (A = 127): exact half-integers round to even; values one ulp
    # either side of a half-integer exercise the near-tie path.
    vals = [127.0, 0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 126.5, -126.5,
            np.nextafter(np.float32(2.5), np.float32(3)), np.nextafter(np.float32(2.5), np.float32(2)),
            np.nextafter(np.float32(-3.5), np.float32(-4)), 3.49999, 3.50001]
    x = np.zeros((1, 1, 1, 64), np.float32)
    x[0, 0, 0, :len(vals)] = vals
    _, q_ref, s_ref = orc.activation_operand(x, "WH", 64)
    q, s = hatq.hatq_fwht_quant_act(dev(x), 1)
    assert np.array_equal(host(s), s_ref) and s_ref[0] == 1.0
    assert_codes(host(q), q_ref, exact=True)
    # a scale that is not a power of two, with quotients near half-integers
    s0 = np.float32(0.37)
    A = np.float32(127) * s0
    ks = np.arange(-60, 60, dtype=np.float32) + np.float32(0.5)
    near = np.concatenate([ks * s0, np.nextafter(ks * s0, np.float32(1e9)),
                           np.nextafter(ks * s0, np.float32(-1e9)), [A]]).astype(np.float32)
    x = near[: (len(near) // 4) * 4].reshape(1, 1, -1, 4)
    _, q_ref, s_ref = orc.activation_operand(x, "WH", 1)
    q, s = hatq.hatq_fwht_quant_act(dev(x), 1)
    assert np.array_equal(host(s), s_ref)
    assert_codes(host(q), q_ref, exact=True)


# ----------------------------------------------------------------------- a1
PREP = [  # (cin, cout, k, stride, pad, form, hblock, transposed, out_pad)
    (128, 128, 1, 1, 0, "DH", 128, False, 0),
    (192, 192, 5, 2, 2, "DH", 64, False, 0),
    (192, 192, 5, 2, 2, "WH", 64, False, 0),
    (192, 192, 5, 2, 2, "DH", 64, True, 1),
    (3, 192, 5, 2, 2, "WH", 64, False, 0),
    (192, 320, 5, 2, 2, "WH", 64, False, 0),
    (64, 64, 3, 2, 1, "WH", 16, True, 1),
    (4, 128, 4, 2, 1, "DH", 4, False, 0),
    (2, 128, 8, 2, 3, "WH", 64, False, 0),
    (4, 64, 5, 2, 2, "WH", 64, False, 0),
]


def _rowrun(cin_p, k, stride, transposed):
    """Geometries whose kernel contracts one 16-byte run per kernel row."""
    return not transposed and cin_p <= 4 and k * cin_p <= 16 and k <= 8 and stride <= 2


@pytest.mark.parametrize("p", PREP, ids=[f"{p[0]}-{p[1]}-k{p[2]}-{p[5]}-b{p[6]}{'-T' if p[7] else ''}" for p in PREP])
def test_prepare_weights_bit_exact(orc, p):
    cin, cout, k, s, pad, form, hb, tr, op = p
    rng = np.random.default_rng(sum(p[:3]))
    w, b = synth.layer_params(rng, cin, cout, k, tr)
    ref = orc.prepare_weights(w, b, cin=cin, cout=cout, k=k, stride=s, pad=pad, form=form,
                              hblock=hb, transposed=tr, out_pad=op)
    layer = hatq.hatq_prepare_weights(hatq.desc(cin, cout, k, s, pad, hb, tr, op), form, dev(w), dev(b))
    assert np.array_equal(unpack_codes(layer, k, ref.cin_p), ref.wq)
    assert np.array_equal(host(layer.w_scale()), ref.w_scale)
    assert np.array_equal(host(layer.bias()), ref.w_bias)
    rr = _rowrun(ref.cin_p, k, s, tr)
    assert layer.w.pack_stride == (-(-16 * k // 64) * 64 if rr else layer.w.k_stride)
    assert np.array_equal(host(layer.wpack()),
                          expected_pack(host(layer.wq()), k, ref.cin_p, rr, layer.w.pack_stride))


def test_pack_weights_rebuilds_copy(orc):
    """hatq_pack_weights after codes written into wq directly."""
    p = PREP[4]
    cin, cout, k, s, pad, form, hb, tr, op = p
    rng = np.random.default_rng(5)
    w, b = synth.layer_params(rng, cin, cout, k, tr)
    layer = hatq.hatq_prepare_weights(hatq.desc(cin, cout, k, s, pad, hb, tr, op), form, dev(w), dev(b))
    wq = synth.int8_codes(rng, (layer.cout_pad, k * k * layer.cin_pad))
    set_codes(layer, wq)
    assert np.array_equal(host(layer.wpack()),
                          expected_pack(host(layer.wq()), k, layer.cin_pad, True, layer.w.pack_stride))


# ----------------------------------------------------------------------- a5
CONV = [  # (n, h, w, cin, cout, k, stride, pad, transposed, out_pad, form, hblock)
    (1, 24, 40, 128, 128, 1, 1, 0, False, 0, "DH", 128),
    (2, 37, 29, 192, 192, 5, 2, 2, False, 0, "DH", 64),
    (2, 37, 29, 192, 192, 5, 2, 2, False, 0, "WH", 64),
    (1, 21, 30, 192, 320, 5, 2, 2, False, 0, "WH", 64),
    (2, 33, 47, 3, 192, 5, 2, 2, False, 0, "WH", 64),
    (1, 9, 13, 192, 192, 5, 2, 2, True, 1, "DH", 64),
    (2, 5, 7, 64, 64, 5, 2, 2, True, 1, "WH", 64),
    (1, 19, 23, 64, 64, 3, 1, 1, False, 0, "DH", 64),
    (1, 17, 15, 64, 256, 3, 2, 1, False, 0, "DH", 64),
    (1, 29, 31, 1, 64, 3, 1, 1, False, 0, "WH", 64),      # row-run, stride 1
    (2, 20, 26, 4, 128, 4, 2, 1, False, 0, "DH", 4),      # row-run, 16-byte runs
    (1, 23, 17, 2, 128, 8, 2, 3, False, 0, "WH", 64),     # row-run, two K-steps
    (1, 21, 19, 3, 320, 5, 2, 2, False, 0, "WH", 64),     # row-run, 64-column tiles
    (1, 18, 22, 4, 64, 5, 2, 2, False, 0, "WH", 64),      # byte-gather path (20-byte runs)
    (1, 30, 70, 192, 192, 4, 2, 1, False, 0, "DH", 64),   # LDS window path, k = 4
    (1, 26, 40, 128, 192, 6, 2, 2, False, 0, "WH", 64),   # LDS window path, k = 6, two chunks
    (2, 20, 21, 64, 192, 5, 2, 2, False, 0, "DH", 64),    # LDS window path, one chunk
    (150, 18, 18, 192, 192, 5, 2, 2, False, 0, "DH", 64), # 300 ragged tiles: blocks walk several, across samples
    (140, 17, 19, 192, 192, 5, 2, 2, False, 0, "WH", 64), # the same, WH
    (150, 18, 18, 64, 192, 5, 2, 2, False, 0, "DH", 64),  # one chunk, 300 tiles (the static tile order)
    (130, 17, 18, 192, 320, 5, 2, 2, False, 0, "WH", 64), # 320 columns: two launches (192 + 128), 260 tiles each
    (3, 21, 30, 192, 320, 5, 2, 2, False, 0, "DH", 64),   # the same split with the DH epilogues
]
CONV_IDS = [f"n{c[0]}-{c[1]}x{c[2]}-{c[3]}to{c[4]}-k{c[5]}s{c[6]}-{c[10]}{'-T' if c[8] else ''}" for c in CONV]


def _layer(orc, c, seed):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng = np.random.default_rng(seed)
    wt, b = synth.layer_params(rng, cin, cout, k, tr)
    ref = orc.prepare_weights(wt, b, cin=cin, cout=cout, k=k, stride=s, pad=p, form=form,
                              hblock=hb, transposed=tr, out_pad=op)
    layer = hatq.hatq_prepare_weights(hatq.desc(cin, cout, k, s, p, hb, tr, op), form, dev(wt), dev(b))
    return rng, wt, b, ref, layer


@pytest.mark.parametrize("c", CONV, ids=CONV_IDS)
def test_conv_int32_bit_exact(orc, c):
    """Identical random INT8 codes on both sides: INT32 accumulators bit-exact."""
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 31)
    xq = synth.int8_codes(rng, (n, h, w, ref.cin_p))
    wq = synth.int8_codes(rng, ref.wq.shape)
    set_codes(layer, wq)
    acc_ref = orc.conv_int8(xq, wq, stride=s, pad=p, transposed=tr, out_pad=op)
    sx = torch.ones(n, device="cuda")
    acc = hatq.hatq_conv_int8(layer, dev(xq), sx, hatq.HATQ_OUT_I32)
    assert np.array_equal(host(acc), acc_ref)


def test_conv_int32_extreme_codes(orc):
    """All +-127 codes: the largest accumulator of the 5x5x192 layers is exact."""
    c = (1, 12, 12, 192, 192, 5, 2, 2, False, 0, "DH", 64)
    rng, wt, b, ref, layer = _layer(orc, c, 32)
    xq = np.full((1, 12, 12, 192), 127, np.int8)
    wq = np.where(rng.random(ref.wq.shape) < 0.5, 127, -127).astype(np.int8)
    wq[0] = 127
    set_codes(layer, wq)
    acc = host(hatq.hatq_conv_int8(layer, dev(xq), torch.ones(1, device="cuda"), hatq.HATQ_OUT_I32))
    acc_ref = orc.conv_int8(xq, wq, stride=2, pad=2)
    assert np.array_equal(acc, acc_ref) and acc.max() == 127 * 127 * 25 * 192


# ----------------------------------------------------------------------- a6
@pytest.mark.parametrize("c", CONV, ids=CONV_IDS)
def test_conv_f32_epilogue(orc, c):
    """The oracle's own codes and scales in, the fp32 output compared:
    DH bit-exact, WH within 1e-6 range-relative."""
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 41)
    x = synth.heavy_tailed_activations(rng, (n, h, w, cin))
    r = orc.layer_forward(x, ref)
    y = host(hatq.hatq_conv_int8(layer, dev(r.xq), dev(r.sx), hatq.HATQ_OUT_F32))
    assert y.shape == r.y.shape
    if form == "DH":
        assert np.array_equal(y, r.y)
    else:
        assert_range_rel(y, r.y)


@pytest.mark.parametrize("c", CONV, ids=CONV_IDS)
def test_layer_forward_exact_inputs(orc, c):
    """Whole layer through hatq_layer_forward on inputs with an exact transform:
    codes identical, so DH is bit-exact and WH within 1e-6."""
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 51)
    x = synth.dyadic_integers(rng, (n, h, w, cin))
    r = orc.layer_forward(x, ref)
    sc = torch.empty(n, device="cuda")
    y = host(hatq.hatq_layer_forward(layer, form, dev(x), act_scale=sc))
    assert np.array_equal(host(sc), r.sx)
    if form == "DH":
        assert np.array_equal(y, r.y)
    else:
        assert_range_rel(y, r.y)


@pytest.mark.parametrize("c", [CONV[1], CONV[2], CONV[4], CONV[5]], ids=[CONV_IDS[i] for i in (1, 2, 4, 5)])
@pytest.mark.parametrize("next_b", [1, 64])
def test_next_absmax(orc, c, next_b):
    """The epilogue's per-sample max |B_next y| equals what the two-pass
    activation kernel computes from the stored y (same fp32 butterfly), and the
    oracle's fp64 value within fp32 rounding."""
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 61)
    x = synth.heavy_tailed_activations(rng, (n, h, w, cin))
    r = orc.layer_forward(x, ref)
    nam = torch.full((n,), -1.0, device="cuda")
    y = hatq.hatq_conv_int8(layer, dev(r.xq), dev(r.sx), hatq.HATQ_OUT_F32, next_hblock=next_b,
                            next_absmax=nam)
    q2, s2 = hatq.hatq_fwht_quant_act(y, next_b)                  # two-pass on the stored y
    q1, s1 = hatq.hatq_fwht_quant_act(y, next_b, absmax=nam)      # single pass with the fused max
    assert torch.equal(s1, s2) and torch.equal(q1, q2)
    S_ref = orc.activation_transform(r.y, next_b).reshape(n, -1)
    A_ref = np.abs(S_ref.astype(np.float64)).max(1)
    np.testing.assert_allclose(host(nam), A_ref, rtol=2e-6)


def test_layer_forward_rejects_form_mismatch(orc):
    c = CONV[1]
    rng, wt, b, ref, layer = _layer(orc, c, 71)
    x = torch.zeros((1, 9, 9, 192), device="cuda")
    with pytest.raises(hatq.HatqError) as e:
        hatq.hatq_layer_forward(layer, "WH", x)
    assert e.value.status == hatq.HATQ_EINVAL
