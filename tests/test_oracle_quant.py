"""Pins for the oracle's symmetric quantizer (Eq. symmetric_q, Eq. current_scale).

Checked against hand-worked examples, the quantizer's defining invariants
(extreme code at the argmax, error at most s/2, odd symmetry, q_max = 2^(8-1)-1),
RNE half-way cases, numpy's own float32 division and rint (a library special
case), and the per-sample reading of the per-tensor scale.
"""
import numpy as np
import pytest

from paper_2608_01653_amd import synth


def test_hand_worked_example(orc):
    # A = 254 -> s = 254/127 = 2 exactly.  S/s = 127, -63.5, 0.25, 0.75, -1.25, 1.5, 2.5
    # RNE: 127, -64 (tie -> even), 0, 1, -1, 2 (tie -> even), 2 (tie -> even)
    S = np.array([[254.0, -127.0, 0.5, 1.5, -2.5, 3.0, 5.0]], np.float32)
    q, s = orc.quantize_symmetric(S)
    assert s[0] == np.float32(2.0)
    assert q.tolist() == [[127, -64, 0, 1, -1, 2, 2]]


def test_ties_to_even_unit_scale(orc):
    # A = 127 -> s = 1 exactly; k + 0.5 rounds to the even neighbour.
    vals = np.array([127.0, 0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 126.5, -126.5], np.float32)
    q, s = orc.quantize_symmetric(vals[None])
    assert s[0] == 1.0
    assert q[0].tolist() == [127, 0, 2, 2, 0, -2, -2, 126, -126]


def test_invariants_heavy_tailed(orc):
    rng = np.random.default_rng(5)
    S = synth.heavy_tailed_activations(rng, (3, 17, 19, 64))
    q, s = orc.quantize_symmetric(S)
    for n in range(3):
        Sn, qn, sn = S[n], q[n].astype(np.int32), np.float64(s[n])
        A = np.abs(Sn).max()
        assert s[n] == np.float32(A / np.float32(127))        # fp32 division of A by 127
        idx = np.unravel_index(np.abs(Sn).argmax(), Sn.shape)
        assert abs(int(qn[idx])) == 127 and np.sign(qn[idx]) == np.sign(Sn[idx])
        assert np.abs(qn).max() <= 127                          # -128 never produced
        err = np.abs(Sn.astype(np.float64) - sn * qn)
        assert err.max() <= sn / 2 * (1 + 1e-6)                # no clamping occurred
    qneg, sneg = orc.quantize_symmetric(-S)
    assert np.array_equal(qneg, -q) and np.array_equal(sneg, s)


def test_matches_numpy_float32(orc):
    rng = np.random.default_rng(6)
    S = synth.heavy_tailed_activations(rng, (2, 33, 64))
    q, s = orc.quantize_symmetric(S)
    for n in range(2):
        A = np.abs(S[n]).max()
        sn = np.float32(A) / np.float32(127.0)
        ref = np.clip(np.rint(S[n] / sn), -127, 127).astype(np.int8)   # float32 / float32
        assert np.array_equal(q[n], ref)


def test_zero_tensor(orc):
    q, s = orc.quantize_symmetric(np.zeros((2, 5, 8), np.float32))
    assert np.all(s == 1.0) and np.all(q == 0)


def test_per_sample_scales_are_independent(orc):
    rng = np.random.default_rng(7)
    a = synth.heavy_tailed_activations(rng, (1, 9, 9, 16))
    b = 1000 * synth.heavy_tailed_activations(rng, (1, 9, 9, 16))
    q1, s1 = orc.quantize_symmetric(a)
    qb, sb = orc.quantize_symmetric(np.concatenate([a, b]))
    assert np.array_equal(qb[0], q1[0]) and sb[0] == s1[0]
