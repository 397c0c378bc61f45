"""Pins for the oracle's group-size rule (Appendix C; Section 3.2).

The paper fixes two limits of the rule, which it prints no data for:
* with very rare failures the optimal group is the whole collaboration,
  m = n (Appendix C: the optimum was m = n in all its experiments);
* with a high enough failure rate it is m = 2 (Section 3.2's decentralized
  SGD case).
Beyond these the rule is the reading stated in oracle/groups.py (parity
unpinned against the paper), checked here against a hand computation and
for the monotonicity the model implies."""

import pytest

from oracle import groups


@pytest.mark.parametrize("n", [2, 3, 8, 16, 64, 300])
def test_no_failures_gives_one_group(n):
    m, e = groups.optimal_group_size(n, 0.0)
    assert m == n and e == 1.0


@pytest.mark.parametrize("n", [4, 16, 64, 300])
def test_high_failure_rate_gives_pairs(n):
    assert groups.optimal_group_size(n, 0.5)[0] == 2
    assert groups.optimal_group_size(n, 0.9)[0] == 2


def test_hand_computed_case():
    # n = 64, p = 0.05: E(2) = 6/0.95^2 = 6.648, E(4) = 3/0.95^4 = 3.684,
    # E(8) = 2/0.95^8 = 3.017, E(16) = 2/0.95^16 = 4.550 (d = 2 for 8..63),
    # E(64) = 1/0.95^64 = 26.6: the optimum is m = 8
    assert groups.iterations(64, 8) == 2 and groups.iterations(64, 7) == 3 and groups.iterations(64, 64) == 1
    m, e = groups.optimal_group_size(64, 0.05)
    assert m == 8 and abs(e - 2 / 0.95 ** 8) < 1e-12


@pytest.mark.parametrize("n", [5, 32, 100])
def test_optimal_size_shrinks_as_failures_grow(n):
    sizes = [groups.optimal_group_size(n, p)[0] for p in (0.0, 0.001, 0.01, 0.03, 0.1, 0.3, 0.6)]
    assert all(a >= b for a, b in zip(sizes, sizes[1:])), sizes
    assert sizes[0] == n and sizes[-1] == 2
