"""Pins for the oracle's weight preparation, epilogues and whole layer (CPU only).

* Function preservation: with quantization switched off, the DH and WH layers equal
  the original float layer (Eq. hadamard_linear_equivalence, Eq.
  weight_only_hadamard_equivalence; padded: Eq. supp_padded_dh, Eq. supp_padded_wh),
  to 1e-5 range-relative.
* Quantization-error bound: the quantized layer stays within the first-order bound
  implied by |x - s q| <= s/2 on both operands (Eq. symmetric_q), which any dropped
  1/b, sign error, transposed transform or misplaced per-channel scale violates.
* b = 1 special case: both forms reduce to plain original-domain W8A8, computed here
  independently with numpy/torch.
* Table I: which transforms sit on each side of a transition, and their
  normalizations.
"""
import os

import numpy as np
import pytest
import scipy.linalg
import torch
import torch.nn.functional as F

from paper_2608_01653_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

LAYERS = [  # (name, n, h, w, cin, cout, k, stride, pad, transposed, out_pad, form, hblock)
    ("1x1_dh_b128", 1, 6, 7, 128, 128, 1, 1, 0, False, 0, "DH", 128),
    ("k5s2_dh_b64", 1, 11, 9, 128, 64, 5, 2, 2, False, 0, "DH", 64),
    ("k5s2_wh_b64", 2, 9, 10, 64, 128, 5, 2, 2, False, 0, "WH", 64),
    ("tconv_dh_b64", 1, 4, 5, 64, 64, 5, 2, 2, True, 1, "DH", 64),
    ("tconv_wh_b64", 1, 4, 3, 32, 64, 5, 2, 2, True, 1, "WH", 64),
    ("rgb_wh_b64", 1, 12, 13, 3, 64, 5, 2, 2, False, 0, "WH", 64),
    ("pad_dh_c40", 1, 7, 6, 40, 16, 3, 1, 1, False, 0, "DH", 64),     # C_in padded 40 -> 64
    ("pad_wh_c40", 1, 7, 6, 16, 40, 3, 1, 1, False, 0, "WH", 64),     # C_out padded 40 -> 64
    ("k5s2_dh_m192", 1, 9, 8, 192, 64, 5, 2, 2, False, 0, "DH", 192),  # H_12 (x) H~_16
    ("k3_wh_m320", 1, 6, 7, 32, 320, 3, 1, 1, False, 0, "WH", 320),    # H_20 (x) H~_16
    ("pad_dh_c17_m20", 1, 7, 6, 17, 8, 3, 1, 1, False, 0, "DH", 20),  # m(17) = 20: Paley-I
    ("pad_wh_c10_m12", 1, 5, 6, 8, 10, 3, 1, 1, False, 0, "WH", 12),  # m(10) = 12
]


def _make(rng, L):
    _, n, h, w, cin, cout, k, s, p, tr, op, form, hb = L
    x = synth.heavy_tailed_activations(rng, (n, h, w, cin))
    wt, b = synth.layer_params(rng, cin, cout, k, tr)
    return x, wt, b


def _prep(orc, L, wt, b, hblock=None):
    _, n, h, w, cin, cout, k, s, p, tr, op, form, hb = L
    return orc.prepare_weights(wt, b, cin=cin, cout=cout, k=k, stride=s, pad=p, form=form,
                               hblock=hblock or hb, transposed=tr, out_pad=op)


def _float(orc, L, x, wt, b):
    _, n, h, w, cin, cout, k, s, p, tr, op, form, hb = L
    xt = torch.from_numpy(x.astype(np.float64)).permute(0, 3, 1, 2)
    wtt = torch.from_numpy(wt.astype(np.float64))
    bt = torch.from_numpy(b.astype(np.float64))
    if tr:
        y = F.conv_transpose2d(xt, wtt, bt, stride=s, padding=p, output_padding=op)
    else:
        y = F.conv2d(xt, wtt, bt, stride=s, padding=p)
    return y.permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("L", LAYERS, ids=[l[0] for l in LAYERS])
def test_unquantized_layer_preserves_function(orc, L):
    rng = np.random.default_rng(11)
    x, wt, b = _make(rng, L)
    pw = _prep(orc, L, wt, b)
    y = orc.layer_unquantized(x, pw)
    ref = _float(orc, L, x, wt, b)
    assert y.shape == ref.shape
    assert np.abs(y - ref).max() <= 1e-5 * np.abs(ref).max()
    # the oracle's own float layer is the same operator
    ref2 = orc.float_layer(x, wt, b, stride=L[7], pad=L[8], transposed=L[9], out_pad=L[10])
    assert np.abs(ref2 - ref).max() <= 1e-12 * np.abs(ref).max()


def _abs_conv(a, wabs, L):
    """sum over taps of a * wabs (both nonnegative), torch float64 (independent)."""
    _, n, h, w, cin, cout, k, s, p, tr, op, form, hb = L
    at = torch.from_numpy(a.astype(np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(wabs.astype(np.float64))          # OHWI
    if tr:
        y = F.conv_transpose2d(at, wt.permute(3, 0, 1, 2), stride=s, padding=p, output_padding=op)
    else:
        y = F.conv2d(at, wt.permute(0, 3, 1, 2), stride=s, padding=p)
    return y.permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("L", LAYERS, ids=[l[0] for l in LAYERS])
def test_quantized_layer_within_error_bound(orc, L):
    rng = np.random.default_rng(12)
    x, wt, b = _make(rng, L)
    _, n, h, w, cin, cout, k, s, p, tr, op, form, hb = L
    pw = _prep(orc, L, wt, b)
    r = orc.layer_forward(x, pw)
    ref = _float(orc, L, x, wt, b)
    sx = r.sx.astype(np.float64)[:, None, None, None]
    What = pw.wq.astype(np.float64) * pw.w_scale.astype(np.float64)[:, None, None, None]
    # accumulator-basis error per channel: (s_x/2) sum|W^| + (s_w,c/2) sum|S|
    ones = np.ones(r.S.shape[:-1] + (r.S.shape[-1],))
    e1 = _abs_conv(ones, np.abs(What), L) * (sx / 2)
    e2 = _abs_conv(np.abs(r.S), np.ones_like(What), L) * (pw.w_scale.astype(np.float64) / 2)
    e = e1 + e2
    if form == "DH":
        bound = e[..., :cout] / hb
    else:
        # |B_b| = 1 entrywise, so the restore spreads each block's errors: sum/b
        blocks = e.reshape(e.shape[:-1] + (-1, hb)).sum(-1, keepdims=True) / hb
        bound = np.broadcast_to(blocks, e.shape[:-1] + (e.shape[-1] // hb, hb))
        bound = bound.reshape(e.shape)[..., :cout]
    slack = 1e-5 * np.abs(ref).max()
    assert np.all(np.abs(r.y - ref) <= bound + slack)
    # and the bound is not vacuous: typical error is well under the signal
    assert np.abs(r.y - ref).mean() < 0.2 * np.abs(ref).mean()


@pytest.mark.parametrize("form", ["DH", "WH"])
def test_block_size_one_is_plain_w8a8(orc, form):
    rng = np.random.default_rng(13)
    L = ("b1", 1, 9, 8, 16, 24, 5, 2, 2, False, 0, form, 1)
    x, wt, b = _make(rng, L)
    pw = _prep(orc, L, wt, b)
    r = orc.layer_forward(x, pw)
    # independent plain W8A8: per-tensor activation scale, per-output-channel weight scale
    sx = np.float32(np.abs(x).max()) / np.float32(127)
    xq = np.clip(np.rint(x / sx), -127, 127)
    wr = wt.astype(np.float32)
    sw = (np.abs(wr).reshape(24, -1).max(1) / np.float32(127)).astype(np.float32)
    wq = np.clip(np.rint(wr / sw[:, None, None, None]), -127, 127)
    acc = F.conv2d(torch.from_numpy(xq).permute(0, 3, 1, 2).double(),
                   torch.from_numpy(wq).double(), stride=2, padding=2).permute(0, 2, 3, 1).numpy()
    ref = acc * (np.float64(sx) * sw.astype(np.float64)) + b.astype(np.float64)
    assert np.array_equal(r.acc.astype(np.float64), acc)
    assert np.abs(r.y - ref).max() <= 2e-7 * np.abs(ref).max()


def test_absorbed_normalization_matches_normalized_codes(orc):
    """Quantizing the unnormalized B x with s~ gives the codes of the normalized
    H x = B x / sqrt(b) with s = s~/sqrt(b) (exact for b = 64, sqrt = 8)."""
    rng = np.random.default_rng(14)
    x = synth.heavy_tailed_activations(rng, (1, 8, 8, 192))
    S, q, s = orc.activation_operand(x, "DH", 64)
    Hn = scipy.linalg.hadamard(64).astype(np.float64) / 8.0
    Sn = (x.astype(np.float64).reshape(-1, 3, 64) @ Hn.T).reshape(S.shape).astype(np.float32)
    assert np.array_equal(Sn * np.float32(8), S)
    sn = np.float32(np.abs(Sn).max()) / np.float32(127)
    assert sn * np.float32(8) == s[0]
    assert np.array_equal(np.clip(np.rint(Sn / sn), -127, 127).astype(np.int8), q)


def _table1():
    rows = {}
    for line in open(os.path.join(GOLDEN, "table1_transitions.txt")):
        if line.strip() and not line.startswith("#"):
            t, go, gi, before, after = line.split()
            rows[t] = (go, gi, before, after)
    return rows


@pytest.mark.parametrize("transition", ["DH-WH", "DH-DH", "WH-WH", "WH-DH"])
def test_table1_transitions(orc, transition):
    """The oracle's epilogue applies the output-side transform exactly when layer l is
    WH, with normalization 1/gamma_out^2 on the unnormalized weights' scale (one
    gamma_out in s_w, one in the restore); the next operand is transformed exactly
    when layer l+1 is DH (Table I, Eq. supp_normalization_factors)."""
    go, gi, before, after = _table1()[transition]
    f_l, f_next = transition.split("-")
    m = 64
    gamma = {"1": 1.0, "sqrt_m": np.sqrt(m)}
    # single nonzero accumulator entry in channel 5 of a 64-channel layer l
    acc = np.zeros((1, 1, 1, m), np.int32)
    acc[..., 5] = 1000
    pw = orc.PreparedWeights(None, np.full(m, 0.5, np.float32), np.zeros(m, np.float32), None,
                             m, m, m, m, 1, 1, 0, False, 0, f_l, m)
    y = orc.epilogue(acc, np.array([0.25], np.float32), pw)[0, 0, 0].astype(np.float64)
    H = scipy.linalg.hadamard(m).astype(np.float64)
    # paper's accumulator scale: s_x * s_w where s_w = s~_w / gamma_out (normalized
    # weights); then H_out = H~/gamma_out restores the basis.  For DH the 1/b of
    # the two input-side normalizations multiplies instead.
    if before == "H":
        g = gamma[go]
        expect = H[:, 5] * (1000 * 0.25 * 0.5 / g) / g
    else:
        assert go == "1"
        expect = np.zeros(m)
        expect[5] = 1000 * 0.25 * 0.5 / m
    np.testing.assert_allclose(y, expect, rtol=1e-7, atol=0)
    # input side of layer l+1
    rng = np.random.default_rng(15)
    xn = synth.dyadic_integers(rng, (1, 2, 2, m))
    S, _, _ = orc.activation_operand(xn, f_next, m)
    if after == "H":
        assert gamma[gi] == np.sqrt(m)
        assert np.array_equal(S.astype(np.float64), xn.astype(np.float64) @ H.T)
    else:
        assert gi == "1" and np.array_equal(S, xn)


@pytest.mark.parametrize("form", ["DH", "WH"])
def test_weight_preparation(orc, form):
    rng = np.random.default_rng(16)
    cin, cout, k = 128, 64, 3
    wt, b = synth.layer_params(rng, cin, cout, k)
    wt[7] = 0.0                                                # an all-zero output row
    pw = orc.prepare_weights(wt, b, cin=cin, cout=cout, k=k, stride=1, pad=1, form=form,
                             hblock=64)
    W = wt.astype(np.float64).transpose(0, 2, 3, 1)           # OHWI
    H = scipy.linalg.hadamard(64).astype(np.float64)
    if form == "DH":
        Wp = (W.reshape(cout, k, k, 2, 64) @ H.T).reshape(W.shape)
        bref = b.astype(np.float64)
    else:
        Wp = np.einsum("ij,jabc->iabc", np.kron(np.eye(1), H), W)
        bref = H @ b.astype(np.float64)
    np.testing.assert_array_equal(pw.w_real, Wp.astype(np.float32))
    np.testing.assert_array_equal(pw.w_bias, bref.astype(np.float32))
    flat = pw.w_real.reshape(cout, -1)
    for c in range(cout):
        A = np.abs(flat[c]).max()
        sc = np.float32(A) / np.float32(127) if A > 0 else np.float32(1)
        assert pw.w_scale[c] == sc
        qc = pw.wq.reshape(cout, -1)[c].astype(np.int32)
        assert np.array_equal(qc, np.clip(np.rint(flat[c] / sc), -127, 127))
        if A > 0:
            assert np.abs(qc).max() == 127
    if form == "DH":
        assert pw.w_scale[7] == 1.0 and not pw.wq[7].any()


@pytest.mark.parametrize("name", ["k5s2_wh_b64", "rgb_wh_b64", "tconv_wh_b64", "k3_wh_m320"])
def test_paired_transition_is_the_accumulator_basis(orc, name):
    """Table I: a WH layer followed by a DH transform of the same blocks gives
    B_next y = z, the dequantized accumulators before the restore (the two
    transforms cancel), up to the fp32 rounding of y and of the transform."""
    L = next(l for l in LAYERS if l[0] == name)
    rng = np.random.default_rng(21)
    x, wt, b = _make(rng, L)
    pw = _prep(orc, L, wt, b)
    r = orc.layer_forward(x, pw)
    z = orc.wh_z(r.acc, r.sx, pw)[..., : pw.cout]
    S = orc.activation_transform(r.y, pw.hblock)
    assert np.abs(S - z).max() <= 2e-6 * np.abs(z).max()
    assert np.abs(S - z).max() > 0 or pw.hblock == 1          # not the same arithmetic
    # the codes: those of z against the oracle's composition, the codes of
    # fl32(B_next y) (Table I with the two transforms explicit), under the code
    # rule (<= 1 LSB on <= 1e-4 of the elements) with scales within 2 ulps
    if pw.hblock > 1:
        qz, sz = orc.quantize_symmetric(z.astype(np.float32))
        qs, ss = orc.quantize_symmetric(S)
        assert np.all(np.abs(sz.astype(np.float64) / ss - 1) <= 2.5e-7)
        d = np.abs(qz.astype(np.int32) - qs.astype(np.int32))
        assert d.max() <= 1 and np.count_nonzero(d) <= 1e-4 * d.size
