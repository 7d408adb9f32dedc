"""The no-allocation entry point hatq_fwht_quant_act_noalloc against the entry
point it varies, hatq_fwht_quant_act (two passes with a caller workspace):
identical codes and scales, bit for bit, on two calls in a row (the second on
a smaller batch, so it must clear what the first left in the shared static
scratch), plus the oracle's codes on exact-transform inputs and the rejection of
batches past the scratch's size."""
import numpy as np
import pytest
import torch

from gpu_util import assert_codes, dev, host
from paper_2608_01653_amd import hatq, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    hatq.load()
    torch.cuda.init()


def _both(x, b):
    n = x.shape[0]
    q_ref, s_ref = hatq.hatq_fwht_quant_act(x, b)
    q = torch.full(x.shape, 99, dtype=torch.int8, device=x.device)
    s = torch.full((n,), -1.0, dtype=torch.float32, device=x.device)
    hatq.hatq_fwht_quant_act_noalloc(x, b, q, s)
    return q, s, q_ref, s_ref


@pytest.mark.parametrize("b", [64, 1, 128])
def test_noalloc_matches_workspace_entry(orc, b):
    rng = np.random.default_rng(500 + b)
    C = 256 if b == 128 else 192
    # first call: a larger batch of heavy-tailed data with a large absmax
    x1 = dev(synth.heavy_tailed_activations(rng, (6, 19, 23, C)) * 100.0)
    q, s, q_ref, s_ref = _both(x1, b)
    assert torch.equal(q, q_ref) and torch.equal(s, s_ref)
    # second call: fewer samples, much smaller values; a stale maximum left in
    # the scratch by the first call would show up as a wrong scale
    x2_np = synth.dyadic_integers(rng, (2, 7, 9, C), lim=64)
    q, s, q_ref, s_ref = _both(dev(x2_np), b)
    assert torch.equal(q, q_ref) and torch.equal(s, s_ref)
    _, q_o, s_o = orc.activation_operand(x2_np, "DH", b)
    assert np.array_equal(host(s), s_o)
    assert_codes(host(q), q_o, exact=True)


def test_noalloc_rejects_past_scratch():
    n = hatq.HATQ_NOALLOC_MAX_SAMPLES + 1
    x = torch.zeros((n, 1, 1, 64), dtype=torch.float32, device="cuda")
    q = torch.zeros((n, 1, 1, 64), dtype=torch.int8, device="cuda")
    s = torch.zeros(n, dtype=torch.float32, device="cuda")
    with pytest.raises(hatq.HatqError) as e:
        hatq.hatq_fwht_quant_act_noalloc(x, 64, q, s)
    assert e.value.status == hatq.HATQ_EUNSUPPORTED
    assert not host(q).any() and not host(s).any()     # nothing launched
