"""The persistent window convolution's tile walk, at sizes with more tiles than
one round of its grid (block b takes the virtual tiles b, b + G, b + 2G, ...,
each refill of a tile's last chunk fetching the next tile's rows): every output
pixel is written by each launch, and launches in a row, launches captured in a
graph and replayed between eager ones, and launches on two streams at once all
give the same int32 accumulators, which match the oracle's direct convolution
on sampled pixels (bit-exact).
"""
import numpy as np
import pytest
import torch

from gpu_util import dev, host
from paper_2608_01653_amd import hatq, synth, workloads

pytestmark = pytest.mark.gpu

SENTINEL = np.iinfo(np.int32).min


def _crop(xq, nb, ih0, iw0, k):
    _, h, w, c = xq.shape
    out = np.zeros((1, k, k, c), np.int8)
    r0, r1 = max(ih0, 0), min(ih0 + k, h)
    c0, c1 = max(iw0, 0), min(iw0 + k, w)
    out[0, r0 - ih0:r1 - ih0, c0 - iw0:c1 - iw0] = xq[nb, r0:r1, c0:c1]
    return out


@pytest.fixture(scope="module")
def case(orc):
    hatq.load()
    torch.cuda.init()
    L = workloads.STACK_B16.layers[1]   # 192 -> 192, 5x5 stride 2 (the window kernel)
    rng = np.random.default_rng(4300)
    w, b = synth.layer_params(rng, L.cin, L.cout, L.k, L.transposed)
    ref = orc.prepare_weights(w, b, cin=L.cin, cout=L.cout, k=L.k, stride=L.stride, pad=L.pad,
                              form=L.form, hblock=L.hblock, transposed=L.transposed, out_pad=L.out_pad)
    d = hatq.desc(L.cin, L.cout, L.k, L.stride, L.pad, L.hblock, L.transposed, L.out_pad)
    layer = hatq.hatq_prepare_weights(d, L.form, dev(w), dev(b))
    # three samples of 512 x 512: 768 tiles of 8 x 32 outputs, three rounds of a
    # 256-block grid
    n, h, wd = 3, 512, 512
    xq = [synth.int8_codes(rng, (n, h, wd, ref.cin_p)) for _ in range(2)]
    sx = torch.full((n,), 0.01, device="cuda")
    return L, ref, layer, xq, sx


def _run(layer, xq_d, sx, y, stream=None):
    return hatq.hatq_conv_int8(layer, xq_d, sx, hatq.HATQ_OUT_I32, y=y, stream=stream)


def _empty(layer, xq):
    n, h, w, _ = xq.shape
    ho, wo = hatq.hatq_conv_out_hw(layer.w.d, h, w)
    return torch.full((n, ho, wo, layer.w.cout_pad), SENTINEL, dtype=torch.int32, device="cuda")


def test_every_pixel_once_and_oracle_samples(orc, case):
    L, ref, layer, xq, sx = case
    y = _run(layer, dev(xq[0]), sx, _empty(layer, xq[0]))
    yh = host(y)
    assert not (yh == SENTINEL).any(), "output pixels not written"
    n, ho, wo, _ = yh.shape
    rng = np.random.default_rng(4301)
    pts = [(s, oh, ow) for s in (0, n - 1) for oh in (0, ho - 1) for ow in (0, wo - 1)]
    pts += [(int(rng.integers(n)), int(rng.integers(ho)), int(rng.integers(wo))) for _ in range(60)]
    for s, oh, ow in pts:
        crop = _crop(xq[0], s, oh * L.stride - L.pad, ow * L.stride - L.pad, L.k)
        acc = orc.conv_int8(crop, ref.wq, stride=L.stride, pad=0)[0, 0, 0]
        assert np.array_equal(yh[s, oh, ow, :L.cout], acc), (s, oh, ow)


def test_launches_in_a_row(case):
    _, _, layer, xq, sx = case
    x0 = dev(xq[0])
    y0 = host(_run(layer, x0, sx, _empty(layer, xq[0])))
    y = _empty(layer, xq[0])
    for i in range(8):
        y.fill_(SENTINEL)
        _run(layer, x0, sx, y)
        assert np.array_equal(host(y), y0), f"launch {i}"


def test_graph_replays(case):
    _, _, layer, xq, sx = case
    x0, x1 = dev(xq[0]), dev(xq[1])
    y0 = host(_run(layer, x0, sx, _empty(layer, xq[0])))
    y1 = host(_run(layer, x1, sx, _empty(layer, xq[1])))
    yg = _empty(layer, xq[0])
    ye = _empty(layer, xq[1])
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _run(layer, x0, sx, yg)   # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        _run(layer, x0, sx, yg)
    for r in range(3):
        yg.fill_(SENTINEL)
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host(yg), y0), f"replay {r}"
        _run(layer, x1, sx, ye)   # eager launches between the replays
        assert np.array_equal(host(ye), y1), f"eager after replay {r}"


def test_two_streams_at_once(case):
    _, _, layer, xq, sx = case
    x0, x1 = dev(xq[0]), dev(xq[1])
    y0 = host(_run(layer, x0, sx, _empty(layer, xq[0])))
    y1 = host(_run(layer, x1, sx, _empty(layer, xq[1])))
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    ya, yb = _empty(layer, xq[0]), _empty(layer, xq[1])
    torch.cuda.synchronize()
    for _ in range(4):
        _run(layer, x0, sx, ya, stream=sa)
        _run(layer, x1, sx, yb, stream=sb)
    torch.cuda.synchronize()
    assert np.array_equal(host(ya), y0)
    assert np.array_equal(host(yb), y1)
