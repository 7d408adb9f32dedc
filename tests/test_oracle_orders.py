"""Pins of the oracle's Hadamard orders beyond powers of two (the supplementary's
Hadamard construction: Paley-I and Paley-II over odd prime powers, Kronecker
products; Eq. hadamard_order, Eq. supp_hadamard_order).

Every constructed matrix has +-1 entries and H H^T = m I.  Paley-I matrices are
skew-Hadamard (H + H^T = 2 I) and Paley-II matrices symmetric, the structure of
the two constructions.  Prime-power fields are pinned twice: by orthogonality
(a wrong quadratic character or field multiplication breaks it) and, for F_9,
by an independent construction over the Gaussian integers modulo 3.  The
order-m matrix is the Kronecker product of its base with a Sylvester matrix,
checked against numpy's kron of scipy's Sylvester matrix.  The order rule is
checked against the supported set enumerated here independently (a prime sieve,
powers generated upward, closure under products), including orders the
constructions do not reach (no existence assumption)."""
import numpy as np
import pytest
import scipy.linalg

import oracle

LIMIT = 4200


def _primes(n):
    sieve = np.ones(n + 1, bool)
    sieve[:2] = False
    for d in range(2, int(n ** 0.5) + 1):
        if sieve[d]:
            sieve[d * d::d] = False
    return np.nonzero(sieve)[0].tolist()


def _odd_prime_powers(n):
    out = set()
    for p in _primes(n):
        if p == 2:
            continue
        v = p
        while v <= n:
            out.add(v)
            v *= p
    return out


def _supported_set(n):
    """Sylvester orders, Paley-I (q + 1, q = 3 mod 4) and Paley-II (2(q + 1),
    q = 1 mod 4) for odd prime powers q, closed under products."""
    pp = _odd_prime_powers(n)
    s = {1 << j for j in range(n.bit_length()) if 1 << j <= n}
    s |= {q + 1 for q in pp if q % 4 == 3}
    s |= {2 * (q + 1) for q in pp if q % 4 == 1 and 2 * (q + 1) <= n}
    while True:
        new = {a * c for a in s for c in s if a * c <= n} - s
        if not new:
            return s
        s |= new


SUPPORTED = _supported_set(LIMIT)


@pytest.mark.parametrize("q,kind", [(3, 1), (7, 1), (11, 1), (19, 1), (23, 1), (31, 1), (43, 1), (191, 1),
                                    (27, 1), (243, 1), (343, 1),
                                    (5, 2), (13, 2), (17, 2), (29, 2), (9, 2), (25, 2), (49, 2), (81, 2),
                                    (121, 2), (125, 2)])
def test_paley_is_hadamard(q, kind):
    H = oracle.paley(q, kind).astype(np.int64)
    m = H.shape[0]
    assert m == (q + 1) * kind
    assert set(np.unique(H)) <= {-1, 1}
    assert np.array_equal(H @ H.T, m * np.eye(m, dtype=np.int64))
    if kind == 1:
        assert np.array_equal(H + H.T, 2 * np.eye(m, dtype=np.int64))     # skew-Hadamard
        Q = H[1:, 1:] - np.eye(q, dtype=np.int64)                          # Jacobsthal core
    else:
        assert np.array_equal(H, H.T)
        Q = None
    if Q is not None:
        # Jacobsthal matrix of F_q: zero diagonal, zero row sums, Q Q^T = q I - J
        assert np.array_equal(np.diag(Q), np.zeros(q, np.int64))
        assert np.array_equal(Q.sum(1), np.zeros(q, np.int64))
        assert np.array_equal(Q @ Q.T, q * np.eye(q, dtype=np.int64) - np.ones((q, q), np.int64))


def test_paley_f9_gaussian_integers():
    """F_9 as the Gaussian integers modulo 3 (i^2 = -1, the smallest monic
    irreducible t^2 + 1): element e = a + 3b is a + b i.  The Paley-II matrix of
    q = 9 built here from the squares of that ring equals the oracle's."""
    elems = [(e % 3, e // 3) for e in range(9)]

    def mul(x, y):
        return ((x[0] * y[0] - x[1] * y[1]) % 3, (x[0] * y[1] + x[1] * y[0]) % 3)

    squares = {mul(x, x) for x in elems if x != (0, 0)}
    assert len(squares) == 4

    def chi(x):
        return 0 if x == (0, 0) else (1 if x in squares else -1)

    n = 10
    C = np.zeros((n, n), np.int64)
    for i in range(n):
        for j in range(n):
            if i == 0 or j == 0:
                C[i, j] = 0 if i == j else 1
            else:
                xi, xj = elems[i - 1], elems[j - 1]
                C[i, j] = chi(((xj[0] - xi[0]) % 3, (xj[1] - xi[1]) % 3))
    zero_blk = np.array([[1, -1], [-1, -1]])
    sign_blk = np.array([[1, 1], [1, -1]])
    H = np.block([[zero_blk if C[i, j] == 0 else C[i, j] * sign_blk for j in range(n)] for i in range(n)])
    assert np.array_equal(oracle.paley(9, 2).astype(np.int64), H)


def test_paley_rejects_wrong_residue():
    for q, kind in [(5, 1), (7, 2), (9, 1), (27, 2), (15, 2), (2, 1), (8, 1), (45, 2), (1, 1)]:
        with pytest.raises(ValueError):
            oracle.paley(q, kind)


def test_every_supported_order_is_hadamard():
    for m in range(1, 401):
        ok = m in SUPPORTED
        assert (oracle.hadamard_base(m) is not None or oracle.hadamard_split(m) is not None) == ok, m
        if ok:
            H = oracle.hadamard(m).astype(np.int64)
            assert np.array_equal(H @ H.T, m * np.eye(m, dtype=np.int64)), m


def test_kronecker_only_order():
    """1904 = 28 * 68 is the smallest order reached only as a product of two
    Paley matrices (no Paley base times a power of two)."""
    extra = sorted(m for m in SUPPORTED if not any(
        m % b == 0 and (m // b) & (m // b - 1) == 0 and (b == 1 or (b - 1 in _odd_prime_powers(b) and (b - 1) % 4 == 3)
                                                      or (b % 2 == 0 and b // 2 - 1 in _odd_prime_powers(b)
                                                          and (b // 2 - 1) % 4 == 1))
        for b in range(1, m + 1)))
    assert extra[0] == 1904
    assert oracle.hadamard_base(1904) is None and oracle.hadamard_split(1904) == 28
    H = oracle.hadamard(1904).astype(np.float64)      # +-1 entries: fp64 sums are exact
    assert np.array_equal(H @ H.T, 1904 * np.eye(1904))
    ref = np.kron(oracle.hadamard(28).astype(np.float64), oracle.hadamard(68).astype(np.float64))
    assert np.array_equal(H, ref)


@pytest.mark.parametrize("m,base,kind,q", [(192, 12, 1, 11), (320, 20, 1, 19), (96, 12, 1, 11), (28, 28, 1, 27),
                                           (12, 12, 1, 11), (128, 1, 0, 0), (52, 52, 2, 25), (100, 100, 2, 49),
                                           (208, 52, 2, 25), (20, 20, 1, 19)])
def test_kronecker_structure(m, base, kind, q):
    b, kk, qq = oracle.hadamard_base(m)
    assert (b, kk, qq) == (base, kind, q)
    P = np.ones((1, 1), np.int64) if b == 1 else oracle.paley(q, kind).astype(np.int64)
    ref = np.kron(P, scipy.linalg.hadamard(m // b).astype(np.int64))
    assert np.array_equal(oracle.hadamard(m).astype(np.int64), ref)


def test_order_rule():
    assert [oracle.order(c) for c in (3, 4, 12, 20, 128, 192, 320)] == [4, 4, 12, 20, 128, 192, 320]
    # prime-power Paley orders: 52 (Paley-II, q = 25) and 100 (Paley-II, q = 49)
    assert [oracle.order(c) for c in (49, 50, 51, 52, 97, 98, 99, 100)] == [52] * 4 + [100] * 4
    assert oracle.order(89) == 96                          # 92 is not reached by these constructions
    with pytest.raises(ValueError):
        oracle.hadamard(92)
    for C in range(1, 1000):
        c4 = 4 * -(-C // 4)
        want = next(m for m in range(c4, LIMIT) if m in SUPPORTED)
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
    # a prime-power order: C = 50 -> one block of 52 (Paley-II over F_25)
    x50 = rng.standard_normal((1, 2, 3, 50)).astype(np.float32)
    S50 = oracle.activation_transform(x50, 52)
    xp = np.concatenate([x50, np.zeros((1, 2, 3, 2), np.float32)], -1).reshape(-1, 52).astype(np.float64)
    ref = (xp @ oracle.paley(25, 2).astype(np.float64).T).astype(np.float32)
    np.testing.assert_allclose(S50.reshape(-1, 52), ref, rtol=0, atol=1e-6 * np.abs(ref).max())
