"""GPU parity of the range-expansion profiling pass (Eq. hadamard_sensitivity):
hatq_range_expansion against the oracle.

* max |x| per sample: bit-exact (a maximum of given values).
* max |S| per sample: the GPU's fp32 butterfly against the oracle's correctly
  rounded dense transform, within 1e-6 of the value (the same fp32 operations
  the quantizer's parity covers).
* The indicator: equal wherever the oracle's margin |max|S|^2 / (b max|x|^2) - 1|
  exceeds 1e-5 (both sides decide exactly in fp64 on their own maxima, which
  can differ in the last bits); inside the margin either answer is valid.
* The count accumulates over calls.
"""
import numpy as np
import pytest
import torch

from gpu_util import dev, host
from paper_2608_01653_amd import hatq, synth

pytestmark = pytest.mark.gpu

MARGIN = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _lib():
    hatq.load()
    torch.cuda.init()


def _inputs(seed, shape):
    rng = np.random.default_rng(seed)
    x = synth.heavy_tailed_activations(rng, shape)
    x[1::2] += np.float32(2.0) * np.abs(x[1::2]).mean()     # a channel mean on every other sample
    return x


def _check(orc, x, b, amax, flags):
    ax, ah, fl = orc.range_expansion(x, b)
    n = x.shape[0]
    am = host(amax)
    assert np.array_equal(am[:n], ax)
    np.testing.assert_allclose(am[n:], ah, rtol=1e-6, atol=0)
    ratio = ah.astype(np.float64) ** 2 / (b * ax.astype(np.float64) ** 2)
    clear = np.abs(ratio - 1) > MARGIN
    assert np.array_equal(host(flags)[clear], fl[clear])
    return fl


CASES = [  # (n, h, w, c, hblock): quad path where c % b == 0 and h*w*c % 4 == 0, else the padded path
    ((6, 9, 11, 64), 64), ((4, 7, 5, 192), 64), ((4, 6, 6, 256), 128), ((4, 5, 9, 192), 1),
    ((6, 13, 7, 32), 8), ((4, 9, 9, 3), 4), ((4, 9, 7, 3), 64), ((4, 5, 7, 5), 2), ((4, 6, 5, 12), 8),
    ((2, 1, 1, 64), 64),
]


@pytest.mark.parametrize("shape,b", CASES, ids=[f"{'x'.join(map(str, s))}-b{b}" for s, b in CASES])
def test_range_expansion_matches_oracle(orc, shape, b):
    x = _inputs(sum(shape) + b, shape)
    xd = dev(x)
    count = torch.zeros(1, dtype=torch.int32, device="cuda")
    amax, flags = hatq.hatq_range_expansion(xd, b, count=count)
    fl = _check(orc, x, b, amax, flags)
    hatq.hatq_range_expansion(xd, b, amax=amax, flags=flags, count=count)     # accumulates
    assert int(host(count)[0]) == 2 * int(host(flags).sum())
    if b == 1:
        assert not fl.any()


@pytest.mark.parametrize("b", [4, 64, 128])
def test_constant_blocks_expand(orc, b):
    """Constant pixel blocks: the butterfly is exact, max|S| = b max|x|."""
    x = np.full((3, 4, 6, 2 * b), 0.75, np.float32)
    x[1] *= -3
    x[2, :, :, b:] = 0
    amax, flags = hatq.hatq_range_expansion(dev(x), b)
    am = host(amax)
    assert np.array_equal(am[3:], b * am[:3]) and host(flags).tolist() == [1, 1, 1]
    _check(orc, x, b, amax, flags)


def test_zero_input():
    x = torch.zeros((2, 4, 4, 64), device="cuda")
    amax, flags = hatq.hatq_range_expansion(x, 64)
    assert not torch.any(amax) and not torch.any(flags)


def test_layer2_input_full_size(orc):
    """The largest activation of the benchmark stack (layer 2's input, 16 x 512 x
    512 x 192 fp32, 3.2 GB): the oracle on the first and last samples, max |x|
    of every sample against torch's reduction, and the count."""
    rng = np.random.default_rng(4300)
    base = synth.heavy_tailed_activations(rng, (1, 512, 512, 192))[0]
    n = 16
    gain = rng.uniform(0.5, 2.0, n).astype(np.float32)
    shift = np.where(np.arange(n) % 2 == 1, np.float32(0.5), np.float32(0.0)).astype(np.float32)
    bd = dev(base)
    xd = torch.empty((n, 512, 512, 192), dtype=torch.float32, device="cuda")
    for k in range(n):
        torch.mul(bd, float(gain[k]), out=xd[k])
        xd[k] += float(shift[k])
    del bd
    count = torch.zeros(1, dtype=torch.int32, device="cuda")
    amax, flags = hatq.hatq_range_expansion(xd, 64, count=count)
    ref_ax = xd.abs().amax(dim=(1, 2, 3))
    assert torch.equal(amax[:n], ref_ax)
    assert int(host(count)[0]) == int(host(flags).sum())
    for k in (0, n - 1):
        xk = (base * gain[k] + shift[k]).astype(np.float32)[None]
        ax, ah, fl = orc.range_expansion(xk, 64)
        am = host(amax)
        assert am[k] == ax[0]
        np.testing.assert_allclose(am[n + k], ah[0], rtol=1e-6, atol=0)
        r = float(ah[0]) ** 2 / (64 * float(ax[0]) ** 2)
        if abs(r - 1) > MARGIN:
            assert int(host(flags)[k]) == int(fl[0])
    del xd
