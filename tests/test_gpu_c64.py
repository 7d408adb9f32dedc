"""The chunk-major code layout [n][c/64][h][w][64] (HATQ_XQ_C64 / HATQ_YQ_C64,
hatq_fwht_quant_act_c64): the same codes as the NHWC layout, placed so the 5x5
stride-2 window kernel's refills read whole 128-byte lines.  Every path is
checked bit for bit against its NHWC twin (Eq. linear_operator: the contraction
does not depend on where each code sits), on ragged tiles and several samples.
"""
import numpy as np
import pytest
import torch

from gpu_util import dev
from paper_2608_01653_amd import hatq, synth, stack, workloads
from test_gpu_parity import _layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    hatq.load()
    torch.cuda.init()


@pytest.mark.parametrize("shape,b", [((2, 9, 11, 192), 64), ((3, 7, 5, 64), 1), ((1, 12, 10, 128), 32),
                                     ((2, 5, 3, 320), 16)])
@pytest.mark.parametrize("given_absmax", [False, True])
def test_quant_c64_equals_nhwc(shape, b, given_absmax):
    rng = np.random.default_rng(101)
    x = dev(synth.heavy_tailed_activations(rng, shape))
    q, s = hatq.hatq_fwht_quant_act(x, b)
    am = (s * 127.0).contiguous() if given_absmax else None
    if given_absmax:
        q, s = hatq.hatq_fwht_quant_act(x, b, absmax=am)
    q64, s64 = hatq.hatq_fwht_quant_act_c64(x, b, absmax=am)
    assert q64.shape == (shape[0], shape[3] // 64, shape[1], shape[2], 64)
    assert torch.equal(s64, s)
    assert torch.equal(hatq.from_c64(q64), q)


WINDOW = [
    (2, 37, 29, 192, 192, 5, 2, 2, False, 0, "DH", 64),
    (3, 21, 30, 192, 320, 5, 2, 2, False, 0, "WH", 64),     # two launches (192 + 128 columns)
    (2, 20, 21, 64, 192, 5, 2, 2, False, 0, "DH", 64),      # one input chunk
    (140, 17, 19, 192, 192, 5, 2, 2, False, 0, "WH", 64),   # ragged tiles across samples
]


@pytest.mark.parametrize("c", WINDOW, ids=[f"n{c[0]}-{c[1]}x{c[2]}-{c[3]}to{c[4]}-{c[10]}" for c in WINDOW])
def test_window_conv_c64_input(orc, c):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 102)
    x = dev(synth.heavy_tailed_activations(rng, (n, h, w, cin)))
    q, sx = hatq.hatq_fwht_quant_act(x, hb if form == "DH" else 1)
    q64 = hatq.to_c64(q)
    # F32 with the fused next-operand absmax
    a1 = torch.full((n,), -1.0, device="cuda")
    a2 = torch.full((n,), -1.0, device="cuda")
    y1 = hatq.hatq_conv_int8(layer, q, sx, hatq.HATQ_OUT_F32, next_hblock=64, next_absmax=a1)
    y2 = hatq.hatq_conv_int8(layer, q64, sx, hatq.HATQ_OUT_F32, next_hblock=64, next_absmax=a2)
    assert torch.equal(y1, y2) and torch.equal(a1, a2)
    # I32 accumulators
    assert torch.equal(hatq.hatq_conv_int8(layer, q, sx, hatq.HATQ_OUT_I32),
                       hatq.hatq_conv_int8(layer, q64, sx, hatq.HATQ_OUT_I32))
    # I8 codes (static scale), NHWC and chunk-major outputs
    if cout % 64 == 0 and cout <= 192:
        sc = (a1 / 127.0).contiguous()
        yq = hatq.hatq_conv_int8(layer, q, sx, hatq.HATQ_OUT_I8, next_hblock=64, out_scale=sc)
        yq64 = hatq.hatq_conv_int8(layer, q64, sx, hatq.HATQ_OUT_I8, next_hblock=64, out_scale=sc, yq_c64=True)
        assert torch.equal(hatq.from_c64(yq64), yq)


@pytest.mark.parametrize("paired", [False, True])
@pytest.mark.parametrize("c", [(3, 45, 141, 3, 192, 5, 2, 2, False, 0, "WH", 64),
                               (40, 9, 11, 3, 192, 5, 2, 2, False, 0, "WH", 64)], ids=["3x45x141", "40x9x11"])
def test_small_cin_codes_c64(orc, c, paired):
    """The small-cin layer's two passes writing the next operand chunk-major."""
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 103)
    x = synth.heavy_tailed_activations(rng, (n, h, w, cin))
    r = orc.layer_forward(x, ref)
    xq, sx = dev(r.xq), dev(r.sx)
    nam = torch.full((n,), -1.0, device="cuda")
    hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32, next_hblock=64, next_absmax=nam, absmax_only=True,
                        paired=paired)
    yq, sq = hatq.hatq_conv_int8_requant(layer, xq, sx, 64, next_absmax=nam, paired=paired)
    yq64, sq64 = hatq.hatq_conv_int8_requant(layer, xq, sx, 64, next_absmax=nam, paired=paired, yq_c64=True)
    assert torch.equal(sq64, sq)
    assert torch.equal(hatq.from_c64(yq64), yq)


@pytest.mark.parametrize("c", [(3, 45, 141, 3, 192, 5, 2, 2, False, 0, "WH", 192)], ids=["3x45x141"])
def test_small_cin_codes_c64_order192(orc, c):
    """The same with the order 192 on both sides (the paper's order for 192
    channels: the 32 x 32 small-cin kernel's order-192 passes)."""
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 104)
    x = synth.heavy_tailed_activations(rng, (n, h, w, cin))
    r = orc.layer_forward(x, ref)
    xq, sx = dev(r.xq), dev(r.sx)
    nam = torch.full((n,), -1.0, device="cuda")
    hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32, next_hblock=192, next_absmax=nam, absmax_only=True)
    yq, sq = hatq.hatq_conv_int8_requant(layer, xq, sx, 192, next_absmax=nam)
    yq64, sq64 = hatq.hatq_conv_int8_requant(layer, xq, sx, 192, next_absmax=nam, yq_c64=True)
    assert torch.equal(sq64, sq)
    assert torch.equal(hatq.from_c64(yq64), yq)
    # and the codes are the two-kernel path's (fp32 output, then the activation kernel)
    y = hatq.hatq_conv_int8(layer, xq, sx, hatq.HATQ_OUT_F32)
    q2, s2 = hatq.hatq_fwht_quant_act(y, 192, absmax=nam)
    assert torch.equal(sq, s2) and torch.equal(yq, q2)


def test_int_transition_c64(orc):
    """The integer transition between two window-kernel layers, both layouts in and out."""
    c = (2, 37, 29, 192, 192, 5, 2, 2, False, 0, "DH", 64)
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, 104)
    x = dev(synth.heavy_tailed_activations(rng, (n, h, w, cin)))
    q, sx = hatq.hatq_fwht_quant_act(x, 64)
    a = torch.empty(n, device="cuda")
    hatq.hatq_conv_int8(layer, q, sx, hatq.HATQ_OUT_F32, next_hblock=64, next_absmax=a)
    table, _ = hatq.hatq_int_transition_params(layer, float(sx.max()), float(a.max()) / 127.0, 64)
    yq = hatq.hatq_conv_int8_int_transition(layer, q, 64, table)
    yq64 = hatq.hatq_conv_int8_int_transition(layer, hatq.to_c64(q), 64, table, yq_c64=True)
    assert torch.equal(hatq.from_c64(yq64), yq)


@pytest.mark.parametrize("paired", [False, True])
def test_stack_step_c64_equals_nhwc(paired):
    """The benchmarked step with chunk-major codes (the default) and with NHWC
    codes: identical codes, scales and output."""
    wl = workloads.ALL["analysis_stack4_rgb_512x768"]
    x_np, params = wl.generate()
    a = stack.Stack(wl, params, c64=True)
    b = stack.Stack(wl, params, c64=False)
    assert any(a.c64) and not any(b.c64)
    x0 = torch.from_numpy(x_np).to(a.dev)
    a.step(x0, paired=paired)
    b.step(x0, paired=paired)
    torch.cuda.synchronize()
    for i in range(a.nL):
        assert torch.equal(a.codes(i), b.codes(i)) and torch.equal(a.sc[i], b.sc[i])
    assert torch.equal(a.output(), b.output())
