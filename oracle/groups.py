"""Group size for the group (Moshpit) all-reduce: TEST INFRASTRUCTURE ONLY.

Appendix C ("Fault tolerance"): the group size m is chosen to minimise the
expected number of iterations needed to reach the global average, counting
both the restarts caused by node failures and the ceil(log_m n) iterations
that groups of m need.  The paper gives no formula (its figure of optimal
sizes prints no data), only two limits: with very rare failures the optimum
is m = n (one global group), and with a high enough failure rate it becomes
m = 2 (Section 3.2, the decentralized-SGD case).

Reading used here: every peer fails independently during one group attempt
with probability p; a group of m succeeds only if none of its members
fails, probability (1 - p)^m, and otherwise restarts, so one iteration takes
1 / (1 - p)^m attempts in expectation; d(m) = ceil(log_m n) iterations are
needed.  E(m) = d(m) / (1 - p)^m, minimised over m in [2, n] (m = n is the
single global group); ties go to the smaller m.  Written as the plain
enumeration of that definition.  Parity unpinned beyond the paper's two
limits: the model of failures is this reading's, not the paper's.
"""

from __future__ import annotations


def iterations(n: int, m: int) -> int:
    """ceil(log_m n): the smallest d >= 1 with m^d >= n."""
    d, reach = 1, m
    while reach < n:
        reach *= m
        d += 1
    return d


def expected_iterations(n: int, m: int, p: float) -> float:
    q = (1.0 - p) ** m  # success probability of one attempt (may underflow to 0)
    return iterations(n, m) / q if q > 0.0 else float("inf")


def optimal_group_size(n: int, p: float, max_group: int = 0):
    """(m, E(m)) minimising the expected iterations over m in
    [2, min(n, max_group or n)]; n >= 2, 0 <= p < 1."""
    best = None
    for m in range(2, min(n, max_group or n) + 1):
        e = expected_iterations(n, m, p)
        if best is None or e < best[1]:
            best = (m, e)
    return best
