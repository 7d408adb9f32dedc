"""Pins of the oracle's integer-only inter-layer transition (Eq. integer_accumulation,
Eq. integer_fixed_point_scale, Eq. integer_hadamard_transition, Table I).

The transition is integer arithmetic, so it is checked against exact rational
arithmetic (Python integers and Fractions, scipy's Sylvester matrices) on small
cases, the fixed-point parameters against their definition, the overflow bound
on extreme codes, and the whole path against the float requantization it
approximates."""
import dataclasses
from fractions import Fraction

import numpy as np
import pytest
import scipy.linalg

import oracle
from paper_2608_01653_amd import synth


def _exact_transition(acc, M, b_int, n, wb, nb, cout):
    """Eq. integer_hadamard_transition with Python integers: v = H_out(M (.) (a + b)),
    w = H_in(v), q = clamp(round(w / 2^n)) with round half to even."""
    P, cout_p = acc.shape
    Ho = scipy.linalg.hadamard(wb).astype(object)
    Hi = scipy.linalg.hadamard(nb).astype(object)
    out = np.zeros((P, cout), np.int8)
    for px in range(P):
        p = [int(M[c]) * (int(acc[px, c]) + int(b_int[c])) for c in range(cout_p)]
        v = []
        for blk in range(0, cout_p, wb):
            v += [sum(Ho[i, j] * p[blk + j] for j in range(wb)) for i in range(wb)]
        v = v[:cout]
        for blk in range(0, cout, nb):
            for i in range(nb):
                w = sum(Hi[i, j] * v[blk + j] for j in range(nb))
                r = round(Fraction(w, 2 ** n))          # Python rounds Fractions half to even
                out[px, blk + i] = max(-127, min(127, r))
    return out


@pytest.mark.parametrize("wb,nb", [(1, 1), (1, 8), (8, 1), (8, 8), (4, 2)])
def test_transition_matches_exact_rationals(wb, nb):
    rng = np.random.default_rng(10 + wb * 3 + nb)
    cout_p = cout = 16
    acc = rng.integers(-300000, 300000, (5, cout_p)).astype(np.int32)
    M = rng.integers(1, 1 << 20, cout_p).astype(np.int32)
    b = rng.integers(-5000, 5000, cout_p).astype(np.int32)
    for n in (0, 1, 7, 30):
        got = oracle.lib()
        q = np.empty((5, cout), np.int8)
        rc = got.orc_int_transition(oracle._p(acc), 5, cout, cout_p, oracle._p(M), oracle._p(b), n, wb, nb,
                                    oracle._p(q))
        assert rc == 0
        assert np.array_equal(q, _exact_transition(acc, M, b, n, wb, nb, cout)), n


def test_round_half_to_even_ties():
    """w / 2^n exactly on a half: even neighbour (both signs)."""
    cout = 1
    M = np.array([1], np.int32)
    b = np.zeros(1, np.int32)
    acc = np.array([[5], [7], [-5], [-7], [4], [6]], np.int32)   # /2 -> 2.5, 3.5, -2.5, -3.5, 2, 3
    q = np.empty((6, 1), np.int8)
    oracle.lib().orc_int_transition(oracle._p(acc), 6, cout, 1, oracle._p(M), oracle._p(b), 1, 1, 1, oracle._p(q))
    assert q.ravel().tolist() == [2, 4, -2, -4, 2, 3]


def _layer(form, hb, seed, cout=64):
    rng = np.random.default_rng(seed)
    w, bias = synth.layer_params(rng, 64, cout, 3, False)
    pw = oracle.prepare_weights(w, bias, cin=64, cout=cout, k=3, stride=1, pad=1, form=form, hblock=hb)
    return rng, pw


@pytest.mark.parametrize("form,next_b", [("DH", 1), ("DH", 64), ("WH", 1), ("WH", 64)])
def test_params_follow_their_definition(form, next_b):
    """u_c = s_x s_w,c / beta_in (one accumulator step), b_int = rne(b / u_c),
    M_c = rne(2^n u_c / (beta_out s_y)), n the largest shift whose multipliers stay
    under the overflow bound; beta_in = 64 for DH, beta_out = 64 for WH."""
    rng, pw = _layer(form, 64, 20)
    s_x, s_y = 0.0123, 0.0456
    rq = oracle.int_requant_params(pw, s_x, s_y, next_b)
    K = pw.k * pw.k * pw.cin_p
    gain = (64 if form == "WH" else 1) * next_b
    sx, sy = Fraction(float(np.float32(s_x))), Fraction(float(np.float32(s_y)))
    bmax = 0
    b_in, b_out = (64, 1) if form == "DH" else (1, 64)
    for c in range(pw.cout_p):
        u = sx * Fraction(float(pw.w_scale[c])) / b_in
        bi = round(Fraction(float(pw.w_bias[c])) / u)
        assert rq.b_int[c] == bi
        bmax = max(bmax, abs(bi))
    mmax = min((1 << 62) // ((K * 127 * 127 + bmax) * gain), (1 << 31) - 1)

    def mults(n):
        return [round(sx * Fraction(float(pw.w_scale[c])) / (b_in * b_out * sy) * 2 ** n) for c in range(pw.cout_p)]
    assert list(rq.M) == mults(rq.shift)
    assert max(mults(rq.shift)) <= mmax < max(mults(rq.shift + 1))


def test_no_overflow_on_extreme_codes():
    """All codes +-127 against the largest multipliers: the int64 sums stay exact
    (compare with Python integers)."""
    rng, pw = _layer("WH", 64, 21)
    rq = oracle.int_requant_params(pw, 0.5, 1e-4, 64)
    K = pw.k * pw.k * pw.cin_p
    acc = np.where(rng.random((2, pw.cout_p)) < 0.5, K * 127 * 127, -K * 127 * 127).astype(np.int32)
    q = oracle.int_transition(acc, pw, rq, 64)
    assert np.array_equal(q, _exact_transition(acc, rq.M, rq.b_int, rq.shift, 64, 64, pw.cout))


@pytest.mark.parametrize("form,next_b", [("DH", 1), ("DH", 64), ("WH", 1), ("WH", 64)])
def test_approximates_float_requantization(form, next_b):
    """Integer codes vs the float path (dequantize, WH restore, next transform,
    quantize with the same static scale).  With the layer's own bias they are at
    most 1 LSB apart (the integer bias rounds b / (s_x s_w) to an integer, up to
    half an accumulator step); with the bias replaced by its integer version
    b_int s_x s_w the float path sees the same accumulator, and the codes differ
    only where M's 2^-24 approximation or fp32 rounding crosses a half."""
    rng, pw = _layer(form, 64, 22)
    x = synth.heavy_tailed_activations(rng, (1, 9, 11, 64))
    S = oracle.activation_transform(x, 64 if form == "DH" else 1)
    s_x = float(np.float32(np.abs(S).max() / 127.0))
    xq = np.clip(np.rint(S / np.float32(s_x)), -127, 127).astype(np.int8)
    acc = oracle.conv_int8(xq, pw.wq, stride=1, pad=1)
    sxv = np.array([s_x], np.float32)

    def float_codes(p, s_y=None):
        y = oracle.epilogue(acc, sxv, p)
        S_next = oracle.activation_transform(y, next_b)
        if s_y is None:
            s_y = float(np.float32(np.abs(S_next).max() / 127.0))
        return np.clip(np.rint(S_next / np.float32(s_y)), -127, 127).astype(np.int32), s_y

    q_float, s_y = float_codes(pw)
    rq = oracle.int_requant_params(pw, s_x, s_y, next_b)
    q_int = oracle.int_transition(acc, pw, rq, next_b).astype(np.int32)
    assert np.abs(q_int - q_float).max() <= 1
    assert np.abs(q_int).max() == 127
    u = np.float64(s_x) * pw.w_scale.astype(np.float64) / (64 if form == "DH" else 1)
    pw_int = dataclasses.replace(pw, w_bias=(rq.b_int.astype(np.float64) * u).astype(np.float32))
    q_float_ib, _ = float_codes(pw_int, s_y)
    d = np.abs(q_int - q_float_ib)
    assert d.max() <= 1 and np.count_nonzero(d) <= 2e-3 * d.size
