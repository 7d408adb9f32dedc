"""Pins of the oracle's Hadamard orders beyond powers of two (the supplementary's
Hadamard construction; Eq. hadamard_order, Eq. supp_hadamard_order).

Every constructed matrix has +-1 entries and H H^T = m I.  Paley-I matrices are
skew-Hadamard (H + H^T = 2 I) and Paley-II matrices symmetric, the structure of
the two constructions.  The order-m matrix is the Kronecker product of its base
with a Sylvester matrix, checked against numpy's kron of scipy's Sylvester
matrix.  The order rule is checked against the supported set enumerated here
independently, including orders the constructions do not reach (no existence
assumption), and the transform of an order-192 block against numpy in fp64."""
import numpy as np
import pytest
import scipy.linalg

import oracle


def _is_prime(q):
    return q >= 2 and all(q % d for d in range(2, int(q ** 0.5) + 1))


def _supported(m):
    bases = {1} | {q + 1 for q in range(3, m + 1) if _is_prime(q) and q % 4 == 3} \
        | {2 * (q + 1) for q in range(5, m + 1) if _is_prime(q) and q % 4 == 1}
    return any(m % b == 0 and (m // b) & (m // b - 1) == 0 for b in bases if b <= m)


@pytest.mark.parametrize("q,kind", [(3, 1), (7, 1), (11, 1), (19, 1), (23, 1), (31, 1), (43, 1), (191, 1),
                                    (5, 2), (13, 2), (17, 2), (29, 2)])
def test_paley_is_hadamard(q, kind):
    H = oracle.paley(q, kind).astype(np.int64)
    m = H.shape[0]
    assert m == (q + 1) * kind
    assert set(np.unique(H)) <= {-1, 1}
    assert np.array_equal(H @ H.T, m * np.eye(m, dtype=np.int64))
    if kind == 1:
        assert np.array_equal(H + H.T, 2 * np.eye(m, dtype=np.int64))     # skew-Hadamard
    else:
        assert np.array_equal(H, H.T)


def test_paley_rejects_wrong_residue():
    for q, kind in [(5, 1), (7, 2), (9, 1), (15, 2), (2, 1)]:
        with pytest.raises(ValueError):
            oracle.paley(q, kind)


def test_every_supported_order_is_hadamard():
    for m in range(1, 401):
        ok = _supported(m)
        assert (oracle.hadamard_base(m) is not None) == ok, m
        if ok:
            H = oracle.hadamard(m).astype(np.int64)
            assert np.array_equal(H @ H.T, m * np.eye(m, dtype=np.int64)), m


@pytest.mark.parametrize("m,base,q", [(192, 12, 11), (320, 20, 19), (96, 12, 11), (28, 28, 13), (12, 12, 11),
                                      (128, 1, 0)])
def test_kronecker_structure(m, base, q):
    b, kind, qq = oracle.hadamard_base(m)
    assert (b, qq) == (base, q)
    P = np.ones((1, 1), np.int64) if b == 1 else oracle.paley(q, kind).astype(np.int64)
    ref = np.kron(P, scipy.linalg.hadamard(m // b).astype(np.int64))
    assert np.array_equal(oracle.hadamard(m).astype(np.int64), ref)


def test_order_rule():
    assert [oracle.order(c) for c in (3, 4, 12, 20, 128, 192, 320)] == [4, 4, 12, 20, 128, 192, 320]
    assert oracle.order(89) == 96                          # 92 is not reached by these constructions
    with pytest.raises(ValueError):
        oracle.hadamard(92)
    for C in range(1, 400):
        c4 = 4 * -(-C // 4)
        want = next(m for m in range(c4, 2000) if _supported(m))
        assert oracle.order(C) == want, C


def test_order192_transform_matches_numpy():
    rng = np.random.default_rng(19)
    x = rng.standard_normal((2, 3, 4, 192)).astype(np.float32)
    S = oracle.activation_transform(x, 192)
    H = np.kron(oracle.paley(11, 1).astype(np.float64), scipy.linalg.hadamard(16))
    ref = (x.reshape(-1, 192).astype(np.float64) @ H.T).astype(np.float32).reshape(S.shape)
    np.testing.assert_allclose(S, ref, rtol=0, atol=1e-6 * np.abs(ref).max())
    # padded: C = 17 -> blocks of 20
    x17 = rng.standard_normal((1, 2, 2, 17)).astype(np.float32)
    S17 = oracle.activation_transform(x17, 20)
    xp = np.concatenate([x17, np.zeros((1, 2, 2, 3), np.float32)], -1).reshape(-1, 20).astype(np.float64)
    np.testing.assert_allclose(S17.reshape(-1, 20), (xp @ oracle.paley(19, 1).astype(np.float64).T),
                               rtol=1e-6, atol=1e-6)
