"""Pins of the oracle's affine activation quantizer (Eq. uniform_q, Eq. affine_q)
and of the convolution on centered codes (Eq. integer_accumulation with a
nonzero activation zero point).

The quantizer runs on the signed grid [-128, 127]; the paper states it on the
unsigned grid [0, 255].  The two give the same scale and codes shifted by 128,
which is checked against the paper's unsigned formulas written with numpy.
Invariants: zero is represented exactly (its code is z), the minimum lands on
q_min, dequantization errs by at most half a step inside the range, one-signed
tensors put z at the grid's end, the all-zero tensor is degenerate.  The
centered convolution is pinned against PyTorch's float64 convolution of x - z
with zero padding (exact on integer data), transposed included."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2608_01653_amd import synth


def _unsigned_paper(S):
    """Eq. affine_q and Eq. uniform_q with q_min = 0, q_max = 255, in numpy float32."""
    lo = np.minimum(S.min(), np.float32(0))
    hi = np.maximum(S.max(), np.float32(0))
    s = np.float32(hi - lo) / np.float32(255)
    z = np.clip(np.rint(np.float32(0) - lo / s), 0, 255)
    q = np.clip(np.rint(S / s) + z, 0, 255)
    return q.astype(np.int32), np.float32(s), int(z)


@pytest.mark.parametrize("seed,shift", [(1, 0.0), (2, 1.5), (3, -2.0), (4, 0.3)])
def test_matches_unsigned_definition(seed, shift):
    rng = np.random.default_rng(seed)
    S = (rng.standard_t(3, (3, 7, 5, 16)) + shift).astype(np.float32)
    q, s, z = oracle.quantize_affine(S)
    for n in range(3):
        qu, su, zu = _unsigned_paper(S[n])
        assert s[n] == su and z[n] == zu - 128
        assert np.array_equal(q[n].astype(np.int32), qu - 128)


def test_invariants():
    rng = np.random.default_rng(7)
    S = (rng.standard_normal((4, 300)) * [[1.0], [3.0], [0.2], [5.0]] + [[0.4], [-1.0], [2.0], [0.0]]).astype(
        np.float32)
    S[:, 17] = 0.0
    q, s, z = oracle.quantize_affine(S)
    for n in range(4):
        qn = q[n].astype(np.int32)
        assert qn[17] == z[n]                                  # zero is exact
        if S[n].min() < 0:
            assert qn[np.argmin(S[n])] == -128                 # the minimum lands on q_min
        assert qn[np.argmax(S[n])] >= 126
        deq = s[n].astype(np.float64) * (qn - z[n])
        err = np.abs(deq - S[n])
        inside = qn < 127
        assert err[inside].max() <= 0.5 * s[n] * (1 + 1e-5)
        assert err.max() <= 1.5 * s[n]


def test_one_signed_and_degenerate():
    pos = np.abs(np.random.default_rng(8).standard_normal((1, 64))).astype(np.float32) + 0.1
    q, s, z = oracle.quantize_affine(pos)
    assert z[0] == -128 and s[0] == np.float32(pos.max()) / np.float32(255)
    q, s, z = oracle.quantize_affine(-pos)
    assert z[0] == 127 and q.min() == -128          # zero (absent here) would sit at the top
    q, s, z = oracle.quantize_affine(np.zeros((2, 10), np.float32))
    assert s.tolist() == [1.0, 1.0] and z.tolist() == [0, 0] and not q.any()


def _torch_conv_centered(xq, z, wq, stride, pad, transposed=False, out_pad=0):
    xc = xq.astype(np.float64) - z[:, None, None, None]
    x = torch.from_numpy(xc).permute(0, 3, 1, 2)
    w = torch.from_numpy(wq.astype(np.float64))
    if transposed:
        y = F.conv_transpose2d(x, w.permute(3, 0, 1, 2), stride=stride, padding=pad, output_padding=out_pad)
    else:
        y = F.conv2d(x, w.permute(0, 3, 1, 2), stride=stride, padding=pad)
    return y.permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("g", [(2, 9, 11, 16, 8, 3, 1, 1), (2, 13, 10, 12, 6, 5, 2, 2), (1, 7, 9, 3, 10, 5, 2, 2)])
def test_centered_conv_matches_torch(g):
    n, h, w, cin, cout, k, s, p = g
    rng = np.random.default_rng(sum(g) + 5)
    xq = synth.int8_codes(rng, (n, h, w, cin))
    wq = synth.int8_codes(rng, (cout, k, k, cin))
    z = rng.integers(-128, 128, n).astype(np.int32)
    acc = oracle.conv_int8(xq, wq, stride=s, pad=p, zx=z)
    assert np.array_equal(acc.astype(np.float64), _torch_conv_centered(xq, z, wq, s, p))
    assert np.array_equal(oracle.conv_int8(xq, wq, stride=s, pad=p, zx=np.zeros(n, np.int32)),
                          oracle.conv_int8(xq, wq, stride=s, pad=p))


def test_centered_transposed_conv_matches_torch():
    rng = np.random.default_rng(11)
    xq = synth.int8_codes(rng, (2, 5, 6, 8))
    wq = synth.int8_codes(rng, (4, 5, 5, 8))
    z = np.array([-100, 37], np.int32)
    acc = oracle.conv_int8(xq, wq, stride=2, pad=2, transposed=True, out_pad=1, zx=z)
    assert np.array_equal(acc.astype(np.float64), _torch_conv_centered(xq, z, wq, 2, 2, True, 1))


def test_centered_width_bound():
    """|x - z| <= 255: 255 * 127 * 25 * 320 = 259,080,000 < 2^31 for the widest layer."""
    assert 255 * 127 * 25 * 320 < 2 ** 31
    xq = np.full((1, 5, 5, 64), 127, np.int8)
    wq = np.full((2, 5, 5, 64), 127, np.int8)
    acc = oracle.conv_int8(xq, wq, stride=1, pad=0, zx=np.array([-128], np.int32))
    assert acc[0, 0, 0, 0] == 255 * 127 * 25 * 64
