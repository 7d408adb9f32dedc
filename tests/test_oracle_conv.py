"""Pins for the oracle's direct INT8 convolution (Eq. integer_accumulation,
Eq. linear_operator): on integer-valued data PyTorch's float64 CPU convolution is
exact, so it is an independent library special case of the same sum.  Covers
1x1, 3x3 and 5x5 kernels, strides 1 and 2, the 5x5 stride-2 transposed
convolution with output padding, ragged spatial sizes and batch > 1, and the
INT32 width bound the supplementary's affine note asks for."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from paper_2608_01653_amd import synth

GEOMS = [  # (n, h, w, cin, cout, k, stride, pad)
    (1, 5, 7, 8, 4, 1, 1, 0),
    (2, 9, 11, 16, 8, 3, 1, 1),
    (1, 13, 10, 12, 6, 5, 2, 2),
    (2, 8, 8, 64, 16, 5, 2, 2),
    (1, 7, 9, 3, 10, 5, 2, 2),
]


def _torch_conv(xq, wq, stride, pad, transposed=False, out_pad=0):
    x = torch.from_numpy(xq.astype(np.float64)).permute(0, 3, 1, 2)
    w = torch.from_numpy(wq.astype(np.float64))           # OHWI
    if transposed:
        # conv_transpose2d wants IOHW: [cin, cout, k, k]
        y = F.conv_transpose2d(x, w.permute(3, 0, 1, 2), stride=stride, padding=pad,
                               output_padding=out_pad)
    else:
        y = F.conv2d(x, w.permute(0, 3, 1, 2), stride=stride, padding=pad)
    return y.permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("g", GEOMS)
def test_conv_int8_matches_torch(orc, g):
    n, h, w, cin, cout, k, s, p = g
    rng = np.random.default_rng(sum(g))
    xq = synth.int8_codes(rng, (n, h, w, cin))
    wq = synth.int8_codes(rng, (cout, k, k, cin))
    acc = orc.conv_int8(xq, wq, stride=s, pad=p)
    ref = _torch_conv(xq, wq, s, p)
    assert acc.dtype == np.int32 and acc.shape == ref.shape
    assert np.array_equal(acc.astype(np.float64), ref)


@pytest.mark.parametrize("h,w,cin,cout", [(4, 6, 8, 4), (5, 3, 16, 8), (1, 1, 4, 4)])
def test_transposed_conv_int8_matches_torch(orc, h, w, cin, cout):
    rng = np.random.default_rng(h * w)
    xq = synth.int8_codes(rng, (2, h, w, cin))
    wq = synth.int8_codes(rng, (cout, 5, 5, cin))
    acc = orc.conv_int8(xq, wq, stride=2, pad=2, transposed=True, out_pad=1)
    assert acc.shape == (2, 2 * h, 2 * w, cout)             # exact 2x upsample
    assert np.array_equal(acc.astype(np.float64), _torch_conv(xq, wq, 2, 2, True, 1))


def test_int32_width_bound(orc):
    """127^2 * 25 * 192 = 77,419,200 < 2^31: the worst case of the largest layer."""
    xq = np.full((1, 5, 5, 192), 127, np.int8)
    wq = np.full((2, 5, 5, 192), 127, np.int8)
    wq[1] = -127
    acc = orc.conv_int8(xq, wq, stride=2, pad=2)
    assert acc[0, 1, 1, 0] == 127 * 127 * 25 * 192 == 77_419_200
    assert acc[0, 1, 1, 1] == -77_419_200
    assert acc.max() < 2**31


@pytest.mark.parametrize("g", GEOMS[:3])
def test_conv_f64_matches_torch(orc, g):
    n, h, w, cin, cout, k, s, p = g
    rng = np.random.default_rng(99 + sum(g))
    x = rng.standard_normal((n, h, w, cin))
    wf = rng.standard_normal((cout, k, k, cin))
    y = orc.conv_f64(x, wf, stride=s, pad=p)
    xt = torch.from_numpy(x).permute(0, 3, 1, 2)
    ref = F.conv2d(xt, torch.from_numpy(wf).permute(0, 3, 1, 2), stride=s, padding=p)
    np.testing.assert_allclose(y, ref.permute(0, 2, 3, 1).numpy(), rtol=1e-12, atol=1e-12)


def test_out_size(orc):
    assert orc.out_size(256, 5, 2, 2) == 128
    assert orc.out_size(255, 5, 2, 2) == 128
    assert orc.out_size(64, 1, 1, 0) == 64
    assert orc.out_size(64, 5, 2, 2, transposed=True, out_pad=1) == 128
