"""GPU parity of the integer-only transition (Eq. integer_accumulation, Eq.
integer_fixed_point_scale, Eq. integer_hadamard_transition, Table I's integer
path): hatq_int_transition_params and hatq_conv_int8_int_transition.

Everything on this path is integer arithmetic once the parameters are fixed,
so the bar is bit-exact throughout:
* the table (M, b_int, n) equals the oracle's for the same prepared weights
  and static scales (both compute it in fp64 with correctly rounded division);
* the codes equal the oracle's integer transition of its own accumulators.
The static scales are per tensor: s_x from the whole batch's transformed
input, s_y from the oracle's float output of the layer (max |B_next y| / 127).
"""
import numpy as np
import pytest
import torch

from gpu_util import assert_codes, dev, host
from paper_2608_01653_amd import hatq, synth, workloads
from test_gpu_parity import CONV, CONV_IDS, _layer
from test_gpu_workloads import _act_block, _crop, _prepare

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    hatq.load()
    torch.cuda.init()


def _static_case(orc, c, next_b, seed):
    n, h, w, cin, cout, k, s, p, tr, op, form, hb = c
    rng, wt, b, ref, layer = _layer(orc, c, seed)
    x = synth.heavy_tailed_activations(rng, (n, h, w, cin))
    S = orc.activation_transform(x, hb if form == "DH" else 1)
    xq, sx = orc.quantize_symmetric(S, per_sample=False)      # one static scale for the batch
    s_x = float(sx[0])
    acc = orc.conv_int8(xq, ref.wq, stride=s, pad=p, transposed=tr, out_pad=op)
    y = orc.epilogue(acc, np.full(n, s_x, np.float32), ref)
    S_next = orc.activation_transform(y, next_b)
    s_y = float(np.float32(np.abs(S_next).max() / np.float32(127.0)))
    return ref, layer, xq, acc, s_x, s_y


@pytest.mark.parametrize("c", CONV, ids=CONV_IDS)
@pytest.mark.parametrize("next_b", [1, 64])
def test_int_transition_bit_exact(orc, c, next_b):
    ref, layer, xq, acc, s_x, s_y = _static_case(orc, c, next_b, 91)
    rq = orc.int_requant_params(ref, s_x, s_y, next_b)
    table, n_shift = hatq.hatq_int_transition_params(layer, s_x, s_y, next_b)
    t = host(table)
    cp = layer.w.cout_pad
    assert n_shift == rq.shift == t[2 * cp]
    assert np.array_equal(t[:cp], rq.M) and np.array_equal(t[cp:2 * cp], rq.b_int)
    q_ref = orc.int_transition(acc, ref, rq, next_b)
    yq = hatq.hatq_conv_int8_int_transition(layer, dev(xq), next_b, table)
    assert yq.shape == q_ref.shape and yq.dtype == torch.int8
    assert_codes(host(yq), q_ref, exact=True, what=f"integer transition next_b={next_b}")
    assert np.abs(q_ref.astype(np.int32)).max() == 127        # the static scale reaches the range end
    # HATQ_PAIRED: B_next B_Cout = b I is exact in integers, so the codes are
    # identical (and for every other layer the flag changes nothing)
    assert torch.equal(hatq.hatq_conv_int8_int_transition(layer, dev(xq), next_b, table, paired=True), yq)


@pytest.mark.parametrize("next_b", [1, 64])
@pytest.mark.parametrize("target", [None, 20, 3])
def test_int_transition_small_shifts_and_reuse(orc, next_b, target):
    """A smaller s_y pushes codes past the range (clamped on both sides) and
    lowers the shift by log2 of the factor with the same multipliers: to 20
    (the general rounding, below 32) and to 3 (below log2 of the block: the WH
    layer whose next operand has the same blocks then shifts left); None
    divides s_y by 8.  The same table serves a second, smaller input."""
    c = CONV[2]
    ref, layer, xq, acc, s_x, s_y = _static_case(orc, c, next_b, 92)
    n1 = orc.int_requant_params(ref, s_x, s_y, next_b).shift
    shrink = 8.0 if target is None else 2.0 ** (n1 - target)
    rq = orc.int_requant_params(ref, s_x, s_y / shrink, next_b)
    assert target is None or rq.shift == target
    table, n_shift = hatq.hatq_int_transition_params(layer, s_x, s_y / shrink, next_b)
    assert n_shift == rq.shift
    assert np.array_equal(host(table)[:layer.w.cout_pad], rq.M)
    q_ref = orc.int_transition(acc, ref, rq, next_b)
    assert np.count_nonzero(np.abs(q_ref.astype(np.int32)) == 127) > 0.01 * q_ref.size
    assert_codes(host(hatq.hatq_conv_int8_int_transition(layer, dev(xq), next_b, table)), q_ref, exact=True)
    assert_codes(host(hatq.hatq_conv_int8_int_transition(layer, dev(xq), next_b, table, paired=True)), q_ref,
                 exact=True)
    small = np.ascontiguousarray(xq[:1, :17, :11])
    acc_s = orc.conv_int8(small, ref.wq, stride=c[6], pad=c[7])
    assert_codes(host(hatq.hatq_conv_int8_int_transition(layer, dev(small), next_b, table)),
                 orc.int_transition(acc_s, ref, rq, next_b), exact=True)


def test_int_params_no_shift_fits(orc):
    """A scale ratio too large for any shift: the table holds n = -1 and zero
    multipliers (the library call itself does not wait; the binding reads the
    shift back and reports it), and a transition with that table writes
    all-zero codes."""
    c = CONV[1]
    _, _, _, _, layer = _layer(orc, c, 93)
    table = torch.zeros(hatq.hatq_int_table_len(layer), dtype=torch.int32, device="cuda")
    with pytest.raises(hatq.HatqError) as e:
        hatq.hatq_int_transition_params(layer, 1.0, 1e-30, 64, table=table)
    assert e.value.status == hatq.HATQ_EUNSUPPORTED
    t = host(table)
    assert t[-1] == -1 and not t[:layer.w.cout_pad].any()
    n, h, w = c[0], c[1], c[2]
    xq = torch.randint(-127, 128, (n, h, w, layer.w.cin_pad), dtype=torch.int8, device="cuda")
    yq = hatq.hatq_conv_int8_int_transition(layer, xq, 64, table)
    assert not host(yq).any()


def test_stack_b16_layer1_int_transition_full_size(orc):
    """The benchmark's layer-1 -> layer-2 transition at full size in integer
    form: sampled pixels bit-exact against the oracle's integer transition of
    its own accumulators, and every code within 1 LSB of the float requantizing
    epilogue at the same static scales (the integer bias and the fixed-point
    multiplier are the only differences)."""
    wl = workloads.STACK_B16
    (ishape, oshape) = wl.shapes()[0]
    L, nxt = wl.layers[0], wl.layers[1]
    rng = np.random.default_rng(4200)
    w, b = synth.layer_params(rng, L.cin, L.cout, L.k, L.transposed)
    ref, layer = _prepare(orc, L, w, b)
    n = ishape[0]
    xq = synth.int8_codes(rng, ishape)
    s_x = 4e-3
    nb = _act_block(nxt)
    xq_d = dev(xq)
    # static s_y from the float pass over the whole batch (fused absmax)
    nam = torch.full((n,), -1.0, device="cuda")
    sx_d = torch.full((n,), s_x, device="cuda")
    hatq.hatq_conv_int8(layer, xq_d, sx_d, hatq.HATQ_OUT_F32, next_hblock=nb, next_absmax=nam, absmax_only=True)
    s_y = float(np.float32(host(nam).max() / np.float32(127.0)))
    table, n_shift = hatq.hatq_int_transition_params(layer, s_x, s_y, nb)
    rq = orc.int_requant_params(ref, s_x, s_y, nb)
    t = host(table)
    cp = layer.w.cout_pad
    assert n_shift == rq.shift and np.array_equal(t[:cp], rq.M) and np.array_equal(t[cp:2 * cp], rq.b_int)
    yq = hatq.hatq_conv_int8_int_transition(layer, xq_d, nb, table)
    assert torch.equal(hatq.hatq_conv_int8_int_transition(layer, xq_d, nb, table, paired=True), yq)
    yf, _ = hatq.hatq_conv_int8_requant(layer, xq_d, sx_d, nb, next_absmax=None,
                                        next_scale=torch.full((n,), s_y, device="cuda"))
    d = (yq.to(torch.int16) - yf.to(torch.int16)).abs()
    assert int(d.max()) <= 1
    del yf, d
    ho, wo = oshape[1], oshape[2]
    pts = [(int(rng.integers(n)), int(rng.integers(ho)), int(rng.integers(wo))) for _ in range(64)]
    pts += [(0, 0, 0), (n - 1, ho - 1, wo - 1)]
    got = host(yq[torch.tensor([p[0] for p in pts]), torch.tensor([p[1] for p in pts]),
                  torch.tensor([p[2] for p in pts])])
    exp = np.empty_like(got)
    for i, (s_, oh, ow) in enumerate(pts):
        crop = _crop(xq, s_, oh * L.stride - L.pad, ow * L.stride - L.pad, L.k)
        acc = orc.conv_int8(crop, ref.wq, stride=L.stride, pad=0)
        exp[i] = orc.int_transition(acc, ref, rq, nb)[0, 0, 0]
    assert_codes(got, exp, exact=True, what="batch-16 stack layer-1 integer transition vs oracle")


@pytest.mark.parametrize("target", [None, 20, 3])
@pytest.mark.parametrize("c", [(3, 45, 141, 3, 192, 5, 2, 2, False, 0, "WH", 64),
                               (40, 9, 11, 3, 192, 5, 2, 2, False, 0, "WH", 64)], ids=["3x45x141", "40x9x11"])
def test_int_transition_small_cin(orc, c, target):
    """The small-cin layer with 192 WH outputs (the RGB input layer; its integer
    transition runs on 32 x 32 MFMA tiles, int64 butterflies, ragged tiles): its
    own shift, 20, and 3 (below log2 of the block: the paired form shifts left);
    bit-exact against the oracle, paired and explicit, NHWC and chunk-major."""
    ref, layer, xq, acc, s_x, s_y = _static_case(orc, c, 64, 94)
    n1 = orc.int_requant_params(ref, s_x, s_y, 64).shift
    shrink = 1.0 if target is None else 2.0 ** (n1 - target)
    rq = orc.int_requant_params(ref, s_x, s_y / shrink, 64)
    assert target is None or rq.shift == target
    table, n_shift = hatq.hatq_int_transition_params(layer, s_x, s_y / shrink, 64)
    assert n_shift == rq.shift
    q_ref = orc.int_transition(acc, ref, rq, 64)
    yq = hatq.hatq_conv_int8_int_transition(layer, dev(xq), 64, table)
    assert_codes(host(yq), q_ref, exact=True, what=f"small-cin integer transition, shift {rq.shift}")
    assert torch.equal(hatq.hatq_conv_int8_int_transition(layer, dev(xq), 64, table, paired=True), yq)
    y64 = hatq.hatq_conv_int8_int_transition(layer, dev(xq), 64, table, yq_c64=True)
    assert torch.equal(hatq.from_c64(y64), yq)
