"""GPU parity of the requantizing epilogue (step a6 with I8 output,
hatq_conv_int8_requant) and of the absmax-only F32 call (y = NULL) that gives
its dynamic scale.

* Against the oracle: the oracle's own layer (codes, scales, fp32 output y_ref)
  fixes S_ref = B_next y_ref and its codes and per-sample scale (Eq.
  symmetric_q, Table I with both transforms explicit); the GPU, fed the
  oracle's codes and scales, must produce the same scale within the bound its
  fp32 butterflies allow and the same codes under the INT8 rule (bit-exact
  where both sides see identical fp32 values: DH layers with next block 1).
* Against the two-kernel GPU path: the codes equal, bit for bit, what the
  activation kernel computes from the stored F32 output with the same absmax
  (same fp32 butterflies, same rounding), and the absmax-only call matches the
  F32 call's fused absmax exactly.  This includes the WH -> DH transition with
  equal blocks, whose WH restore and next butterfly both run.
* HATQ_PAIRED: a WH layer whose next operand uses the same blocks takes the
  next operand as z, the accumulators dequantized before the restore (B_next y
  = z in exact arithmetic, Table I): scale and codes bit for bit against the
  oracle's z, and within the code rule against the oracle's composition (codes
  of fl32(B_next y_ref)).  For every other layer the flag changes nothing.
* A static scale (next_absmax = NULL) gives the oracle's codes for that scale,
  through hatq_conv_int8_requant and through hatq_conv_int8 in I8 mode.
"""
import numpy as np
import pytest
import torch

from gpu_util import assert_codes, assert_scale_ulp, dev, host
from paper_2608_01653_amd import hatq, synth
from test_gpu_parity import CONV, CONV_IDS, _layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    hatq.load()
    torch.cuda.init()


def _oracle_next(orc, r, next_b):
    S_ref = orc.activation_transform(r.y, next_b)
    q_ref, s_ref = orc.quantize_symmetric(S_ref)
    return q_ref, s_ref


def _paired(c, next_b):
    """A WH layer whose next operand uses the same blocks (the HATQ_PAIRED case)."""
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    return form == "WH" and next_b == hb and hb > 1 and cout % hb == 0


def _gamma(k):
    u = 2.0 ** -24
    return k * u / (1 - k * u)


def _scale_tol(orc, r, ref, next_b, s_ref, form):
    """Bound on |s_gpu - s_ref| for the scale of B_next y.  The GPU forms B_next y
    with log2(b) rounded fp32 butterfly stages (the oracle in fp64 with one
    rounding), so each value differs by at most gamma_k * (sum of |y| over its
    block).  A WH layer's y itself differs from the oracle's: the GPU restores
    z / b (exact) with six rounded stages, the oracle rounds (B z) / b once, so
    |dy| <= gamma_6 * (sum of |z| over the restored block) / b + u |y|; a value
    of the next operand sums next_b of them.  The maxima differ by at most the
    largest value difference; over 127, plus two ulps (the roundings of both
    scales and of the oracle's transformed values)."""
    n = r.y.shape[0]
    k = int(np.log2(next_b)) if next_b > 1 else 0
    ya = np.abs(r.y.astype(np.float64))
    ya = np.pad(ya, [(0, 0)] * 3 + [(0, (-ya.shape[-1]) % next_b)])
    tol = _gamma(k) * ya.reshape(n, -1, next_b).sum(-1).max(-1)
    if form == "WH":
        hb = ref.hblock
        za = np.abs(orc.wh_z(r.acc, r.sx, ref).astype(np.float64))
        dy = _gamma(int(np.log2(hb))) * za.reshape(n, -1, hb).sum(-1).max(-1) / hb
        dy = dy + 2.0 ** -24 * np.abs(r.y.astype(np.float64)).reshape(n, -1).max(-1)
        tol = tol + max(next_b, 1) * dy
    return tol / 127 + 2 * np.spacing(s_ref.astype(np.float32)).astype(np.float64)


@pytest.mark.parametrize("c", CONV, ids=CONV_IDS)
@pytest.mark.parametrize("next_b", [1, 64])
def test_requant_codes(orc, c, next_b):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 81)
    x = synth.heavy_tailed_activations(rng, (n, h, w, cin))
    r = orc.layer_forward(x, ref)
    q_ref, s_ref = _oracle_next(orc, r, next_b)
    xq, sx = dev(r.xq), dev(r.sx)
    # pass 1: the absmax alone; pass 2: the codes (both transforms explicit)
    nam = torch.full((n,), -1.0, device="cuda")
    assert hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32, next_hblock=next_b, next_absmax=nam,
                               absmax_only=True) is None
    yq, sq = hatq.hatq_conv_int8_requant(layer, xq, sx, next_b, next_absmax=nam)
    assert yq.shape == q_ref.shape and yq.dtype == torch.int8
    if form == "DH" and next_b == 1:
        assert_scale_ulp(host(sq), s_ref)
        assert_codes(host(yq), q_ref, exact=True, what=f"requant codes next_b={next_b}")
    else:
        tol = _scale_tol(orc, r, ref, next_b, s_ref, form)
        assert np.all(np.abs(host(sq).astype(np.float64) - s_ref) <= tol), (host(sq), s_ref, tol)
        assert_codes(host(yq), q_ref, exact=False, what=f"requant codes next_b={next_b}")
    # the two-kernel GPU path on the stored output: identical absmax, scale and codes
    nam2 = torch.full((n,), -1.0, device="cuda")
    y = hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32, next_hblock=next_b, next_absmax=nam2)
    q2, s2 = hatq.hatq_fwht_quant_act(y, next_b, absmax=nam2)
    assert torch.equal(nam, nam2)
    assert torch.equal(sq, s2)
    assert torch.equal(yq, q2)
    # the same two passes with HATQ_PAIRED
    namp = torch.full((n,), -1.0, device="cuda")
    hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32, next_hblock=next_b, next_absmax=namp,
                        absmax_only=True, paired=True)
    yqp, sqp = hatq.hatq_conv_int8_requant(layer, xq, sx, next_b, next_absmax=namp, paired=True)
    if _paired(c, next_b):
        qz, sz = orc.quantize_symmetric(orc.wh_z(r.acc, r.sx, ref)[..., :cout])
        # the same fp32 z on both sides: scale and codes bit for bit
        assert np.array_equal(host(sqp), sz)
        assert_codes(host(yqp), qz, exact=True, what=f"paired requant codes next_b={next_b}")
        # and the oracle's composition within the code rule
        assert np.all(np.abs(host(sqp).astype(np.float64) - s_ref) <= _scale_tol(orc, r, ref, next_b, s_ref, form))
        assert_codes(host(yqp), q_ref, what="paired requant codes vs the oracle's composition")
    else:
        assert torch.equal(namp, nam) and torch.equal(sqp, sq) and torch.equal(yqp, yq)


@pytest.mark.parametrize("ci", [1, 2, 4, 5, 16], ids=[CONV_IDS[i] for i in (1, 2, 4, 5, 16)])
def test_requant_static_scale(orc, ci):
    c = CONV[ci]
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 82)
    x = synth.heavy_tailed_activations(rng, (n, h, w, cin))
    r = orc.layer_forward(x, ref)
    q_ref, s_ref = _oracle_next(orc, r, 64)
    sc = dev(s_ref.copy())
    yq, sq = hatq.hatq_conv_int8_requant(layer, dev(r.xq), dev(r.sx), 64, next_absmax=None, next_scale=sc)
    assert np.array_equal(host(sq), s_ref)      # an input: left as given
    assert_codes(host(yq), q_ref, what="requant codes, static scale")
    # hatq_conv_int8 in I8 mode with out_scale: the same kernel, the same codes
    y8 = hatq.hatq_conv_int8(layer, dev(r.xq), dev(r.sx), hatq.HATQ_OUT_I8, next_hblock=64, out_scale=sc)
    assert y8.dtype == torch.int8 and torch.equal(y8, yq)
    assert np.array_equal(host(sc), s_ref)


def test_requant_zero_output():
    """All-zero codes and bias: absmax 0 gives scale 1 and all-zero codes."""
    c = CONV[1]
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    layer = hatq.hatq_prepare_weights(hatq.desc(cin, cout, k, s, p, hb, tr, op), form,
                                      torch.randn(cout, cin, k, k, device="cuda"), torch.zeros(cout, device="cuda"))
    xq = torch.zeros((n, h, w, cin), dtype=torch.int8, device="cuda")
    sx = torch.ones(n, device="cuda")
    nam = torch.full((n,), -1.0, device="cuda")
    hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32, next_hblock=64, next_absmax=nam, absmax_only=True)
    yq, sq = hatq.hatq_conv_int8_requant(layer, xq, sx, 64, next_absmax=nam)
    assert torch.all(nam == 0) and torch.all(sq == 1) and not torch.any(yq)


@pytest.mark.gpu
def test_codes_into_4_byte_aligned_buffers(orc):
    """Code outputs at an address that is 4- but not 16-byte aligned (all the ABI
    asks of them): the activation quantizer and the requantizing epilogue write
    the same codes as into aligned buffers."""
    rng = np.random.default_rng(91)
    x = dev(synth.heavy_tailed_activations(rng, (2, 9, 11, 192)))
    q_ref, s_ref = hatq.hatq_fwht_quant_act(x, 64)
    buf = torch.zeros(q_ref.numel() + 32, dtype=torch.int8, device="cuda")
    q_off = buf[4:4 + q_ref.numel()].view(q_ref.shape)
    q_got, s_got = hatq.hatq_fwht_quant_act(x, 64, xq=q_off)
    assert q_off.data_ptr() % 16 == 4
    assert torch.equal(q_got, q_ref) and torch.equal(s_got, s_ref)
    assert torch.equal(buf[:4], torch.zeros(4, dtype=torch.int8, device="cuda"))
    assert torch.equal(buf[4 + q_ref.numel():], torch.zeros(28, dtype=torch.int8, device="cuda"))
    # samples of 84 elements (one full item of 64 and a tail): every sample after
    # the first starts 4, 8 or 12 bytes past a 16-byte boundary (original-domain
    # codes, exact on both sides)
    xs = synth.heavy_tailed_activations(rng, (5, 4, 7, 3))
    q_small, _ = hatq.hatq_fwht_quant_act(dev(xs), 1)
    q_exp, _ = orc.quantize_symmetric(xs)
    assert np.array_equal(host(q_small), q_exp)

    c = (2, 21, 23, 192, 192, 5, 2, 2, False, 0, "DH", 64)
    _, _, _, _, layer = _layer(orc, c, 92)
    nam = torch.full((2,), -1.0, device="cuda")
    assert hatq.hatq_conv_int8(layer, q_ref, s_ref, hatq.HATQ_OUT_F32, next_hblock=64, next_absmax=nam,
                               absmax_only=True) is None
    y_ref, _ = hatq.hatq_conv_int8_requant(layer, q_ref, s_ref, 64, next_absmax=nam)
    ybuf = torch.zeros(y_ref.numel() + 32, dtype=torch.int8, device="cuda")
    y_off = ybuf[4:4 + y_ref.numel()].view(y_ref.shape)
    y_got, _ = hatq.hatq_conv_int8_requant(layer, q_ref, s_ref, 64, next_absmax=nam, yq=y_off)
    assert y_off.data_ptr() % 16 == 4
    assert torch.equal(y_got, y_ref)
    assert torch.equal(ybuf[4 + y_ref.numel():], torch.zeros(28, dtype=torch.int8, device="cuda"))


# The small-cin layer with 192 WH outputs into a next operand with blocks of 64
# (the RGB input layer of the analysis transform): its two passes run on 32 x 32
# MFMA tiles of 8 output rows x 32 columns.  Ragged tiles in both directions,
# k = 6, stride 1, and many one-tile samples.
SMALL_CIN = [
    (3, 45, 141, 3, 192, 5, 2, 2, False, 0, "WH", 64),
    (2, 30, 40, 3, 192, 6, 2, 2, False, 0, "WH", 64),
    (1, 20, 70, 3, 192, 5, 1, 2, False, 0, "WH", 64),
    (40, 9, 11, 3, 192, 5, 2, 2, False, 0, "WH", 64),
]


@pytest.mark.parametrize("c", SMALL_CIN, ids=[f"n{c[0]}-{c[1]}x{c[2]}-k{c[5]}s{c[6]}" for c in SMALL_CIN])
def test_requant_small_cin_tiles(orc, c):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 83)
    x = synth.heavy_tailed_activations(rng, (n, h, w, cin))
    r = orc.layer_forward(x, ref)
    q_ref, s_ref = _oracle_next(orc, r, 64)
    xq, sx = dev(r.xq), dev(r.sx)
    nam = torch.full((n,), -1.0, device="cuda")
    assert hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32, next_hblock=64, next_absmax=nam,
                               absmax_only=True) is None
    yq, sq = hatq.hatq_conv_int8_requant(layer, xq, sx, 64, next_absmax=nam)
    tol = _scale_tol(orc, r, ref, 64, s_ref, form)
    assert np.all(np.abs(host(sq).astype(np.float64) - s_ref) <= tol), (host(sq), s_ref, tol)
    assert_codes(host(yq), q_ref, exact=False, what="small-cin requant codes")
    # the F32 output with its fused absmax, then the activation kernel: the same
    # absmax, scale and codes bit for bit
    nam2 = torch.full((n,), -1.0, device="cuda")
    y = hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32, next_hblock=64, next_absmax=nam2)
    q2, s2 = hatq.hatq_fwht_quant_act(y, 64, absmax=nam2)
    assert torch.equal(nam, nam2)
    assert torch.equal(sq, s2)
    assert torch.equal(yq, q2)
    # HATQ_PAIRED: the next operand is z itself (no transform): scale and codes
    # bit for bit against the oracle's z, and within the code rule against its
    # composition
    namp = torch.full((n,), -1.0, device="cuda")
    hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32, next_hblock=64, next_absmax=namp, absmax_only=True,
                        paired=True)
    yqp, sqp = hatq.hatq_conv_int8_requant(layer, xq, sx, 64, next_absmax=namp, paired=True)
    qz, sz = orc.quantize_symmetric(orc.wh_z(r.acc, r.sx, ref)[..., :cout])
    assert np.array_equal(host(sqp), sz)
    assert_codes(host(yqp), qz, exact=True, what="paired small-cin codes")
    assert np.all(np.abs(host(sqp).astype(np.float64) - s_ref) <= tol)
    assert_codes(host(yqp), q_ref, what="paired small-cin codes vs the oracle's composition")
