"""Pins of the oracle's range-expansion statistic (Eq. hadamard_sensitivity) and
the DH/WH rule (Eq. layerwise_hadamard_selection).

The statistic compares the orthonormal transform H = B / sqrt(b) of a sample
with the sample itself in the infinity norm.  Closed forms: a constant pixel
block is mapped onto the constant Hadamard basis (Eq.
hadamard_mean_accumulation: sqrt(b) times the channel mean, an expansion); a
one-hot block spreads evenly (1/sqrt(b) of the peak, no expansion); two equal
entries of a block of 4 land exactly on the boundary (not an expansion, the
comparison is strict).  Brute force against scipy's Sylvester matrices in fp64
on small tensors, padding included."""
import numpy as np
import pytest
import scipy.linalg

import oracle


def _brute(x, b):
    """fp64 reference: (max |x|, max |B x_pad| rounded to fp32, exact-margin ratio)."""
    n, C = x.shape[0], x.shape[-1]
    Cp = -(-C // b) * b
    xp = np.zeros(x.shape[:-1] + (Cp,), np.float64)
    xp[..., :C] = x
    H = scipy.linalg.hadamard(b).astype(np.float64)
    S = (xp.reshape(-1, Cp // b, b) @ H.T).reshape(n, -1)
    ax = np.abs(x.reshape(n, -1)).max(axis=1)
    ah = np.abs(S).max(axis=1)
    return ax.astype(np.float32), ah.astype(np.float32), ah / (np.sqrt(b) * ax.astype(np.float64))


@pytest.mark.parametrize("b", [2, 4, 8, 16, 32, 64, 128])
def test_constant_block_expands(b):
    mu = np.float32(0.375)
    x = np.full((2, 3, 5, 2 * b), mu, np.float32)
    x[1] *= -2
    ax, ah, fl = oracle.range_expansion(x, b)
    assert np.array_equal(ax, np.abs(x.reshape(2, -1)).max(axis=1))
    assert np.array_equal(ah, b * ax)                     # the constant basis collects the whole block
    assert fl.tolist() == [1, 1]


@pytest.mark.parametrize("b", [2, 4, 8, 64])
def test_one_hot_block_does_not_expand(b):
    x = np.zeros((1, 4, 4, b), np.float32)
    x[0, :, :, 1] = 1.0
    x[0, 2, 3, 1] = -3.0
    ax, ah, fl = oracle.range_expansion(x, b)
    assert ax[0] == 3.0 and ah[0] == 3.0 and fl[0] == 0


def test_boundary_is_not_an_expansion():
    """Two equal entries in a block of 4: |H x| / 2 = (2, 0, 2, 0) / 2 = x's peak."""
    x = np.zeros((2, 1, 1, 4), np.float32)
    x[0, 0, 0, :2] = 1.0
    x[1, 0, 0, :3] = 1.0                                   # three: (3, 1, 1, -1) / 2 > 1
    ax, ah, fl = oracle.range_expansion(x, 4)
    assert ah.tolist() == [2.0, 3.0] and fl.tolist() == [0, 1]


def test_identity_block_never_expands():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((3, 5, 7, 6)).astype(np.float32)
    ax, ah, fl = oracle.range_expansion(x, 1)
    assert np.array_equal(ax, ah) and not fl.any()


@pytest.mark.parametrize("shape,b", [((4, 6, 5, 64), 64), ((3, 9, 9, 3), 4), ((5, 7, 3, 12), 8),
                                     ((2, 5, 5, 192), 64), ((4, 3, 3, 5), 2)])
def test_matches_brute_force(shape, b):
    rng = np.random.default_rng(sum(shape) + b)
    x = rng.standard_t(3, shape).astype(np.float32)
    x[1::2] += np.float32(1.5)                            # a channel mean on every other sample
    ax, ah, fl = oracle.range_expansion(x, b)
    rax, rah, ratio = _brute(x, b)
    assert np.array_equal(ax, rax)
    np.testing.assert_allclose(ah, rah, rtol=1e-7)
    clear = np.abs(ratio - 1) > 1e-6
    assert clear.all()
    assert np.array_equal(fl.astype(bool), ratio > 1)


def test_select_form_rule():
    assert oracle.select_form(800, 1000, 0.8) == "DH"     # p = tau: DH (strict inequality)
    assert oracle.select_form(801, 1000, 0.8) == "WH"
    assert oracle.select_form(0, 1, 0.8) == "DH" and oracle.select_form(1, 1, 0.8) == "WH"
    assert oracle.select_form(4, 5, 0.8) == "DH" and oracle.select_form(5, 6, 0.8) == "WH"
    for bad in [(1, 0), (-1, 4), (5, 4)]:
        with pytest.raises(ValueError):
            oracle.select_form(*bad)


@pytest.mark.parametrize("b", [12, 20, 52, 192])
def test_kronecker_orders_statistic(orc, b):
    """The statistic with the paper's non-power-of-two orders (the supplementary
    Hadamard construction).  Paley-I matrices (q + 1 = 12, 20; 192 = P_12 (x)
    H~_16) have an all-ones first row, so a constant block lands on it (max|S|
    = b|c|, an expansion); for every order a one-hot block gives a column of
    +-1 entries (max|S| = |x|, no expansion), and a random input equals the
    dense transform by numpy with the same matrix."""
    H = orc.hadamard(b).astype(np.float64)
    if orc.hadamard_base(b)[1] != 2:                   # Paley-I based
        assert np.all(H[0] == 1)
        x = np.full((1, 2, 3, b), -0.75, np.float32)
        ax, ah, fl = orc.range_expansion(x, b)
        assert ah[0] == np.float32(0.75 * b) and fl[0] == 1
    e = np.zeros((1, 1, 1, b), np.float32)
    e[0, 0, 0, b // 3] = 2.5
    ax, ah, fl = orc.range_expansion(e, b)
    assert ax[0] == 2.5 and ah[0] == 2.5 and fl[0] == 0
    rng = np.random.default_rng(b)
    x = rng.standard_normal((2, 3, 4, 2 * b)).astype(np.float32)
    ax, ah, fl = orc.range_expansion(x, b)
    S = (x.reshape(2, -1, b).astype(np.float64) @ H.T).astype(np.float32)
    np.testing.assert_array_equal(ah, np.abs(S).reshape(2, -1).max(1))
    np.testing.assert_array_equal(fl, (ah.astype(np.float64) ** 2 > b * ax.astype(np.float64) ** 2).astype(np.int32))
