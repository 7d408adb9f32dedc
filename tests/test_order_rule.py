"""The library's transform order rule (hatq_hadamard_order, Eq. hadamard_order
with the supplementary Hadamard construction) against the oracle's, which is
pinned on its own in test_oracle_orders.py: the same m(C) for every channel
count up to 1024 and on a sample up to the 4096 limit, the values the paper's
workloads use, and the limits.  Host only (no GPU)."""
import pytest

from paper_2608_01653_amd import hatq


@pytest.fixture(scope="module")
def L():
    return hatq.load(build_if_missing=True)


def test_order_rule_matches_oracle(L, orc):
    cs = list(range(1, 1025)) + list(range(1025, 4097, 37)) + [4093, 4096]
    for c in cs:
        assert hatq.hatq_hadamard_order(c) == orc.order(c), c


def test_order_rule_values(L):
    # the workloads' channel counts (RGB, 128, 192, 320), and orders whose only
    # construction is Paley-II over a prime power: 52 = 2 (25 + 1), q = 5^2, and
    # 100 = 2 (49 + 1), q = 7^2
    expect = {1: 4, 3: 4, 4: 4, 5: 8, 9: 12, 128: 128, 192: 192, 320: 320, 49: 52, 52: 52, 97: 100, 100: 100}
    for c, m in expect.items():
        assert hatq.hatq_hadamard_order(c) == m, c
    assert hatq.hatq_hadamard_order(0) == 0 and hatq.hatq_hadamard_order(4097) == 0
