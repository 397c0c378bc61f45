"""Pins for the oracle's load-balancing LP (Appendix B; Eq. main_problem and
its relaxation).  Its solver is scipy's HiGHS; what is pinned is the LP it
builds:

* compute-bound collaborations reach xi = sum(s)/B (closed form);
* homogeneous peers that all compute reach the all-reduce rate
  xi = n*b / (2*(n-1)*P) (Section 3.2's AR-SGD special case, closed form),
  with b the narrower of download and upload when they differ;
* with compute to spare, the relaxation reaches its bound xi = 2*b/P: the
  return to oneself g_ii is limited only through (1 - c_k)*d_i, so as c -> 0
  each peer receives d_i from itself plus d_i over the network (closed form
  of the relaxed LP, which the binary problem cannot reach);
* the relaxation bounds every binary choice of c from above (brute force
  over c in {0,1}^n, n <= 4);
* the returned solution satisfies every constraint, and its shares sum to 1."""

import itertools

import numpy as np
import pytest

from oracle import lp


@pytest.mark.parametrize("n", [2, 3, 5])
def test_compute_bound(n):
    s = np.full(n, 100.0)
    b = np.full(n, 1e12)
    r = lp.solve(s, b, b, B=4096.0, P=1e6)
    assert np.isclose(r["xi"], n * 100.0 / 4096.0, rtol=1e-7)
    assert lp.violation(r, s, b, b, 4096.0, 1e6) < 1e-7


@pytest.mark.parametrize("n", [2, 3, 4, 8])
def test_all_reduce_rate_when_all_compute(n):
    s = np.full(n, 1e9)
    b = np.full(n, 1e6)
    P = 2e6
    r = lp.solve(s, b, b, B=1.0, P=P, fix_c=np.ones(n))
    assert np.isclose(r["xi"], n * 1e6 / (2 * (n - 1) * P), rtol=1e-6)
    assert np.isclose(r["frac"].sum(), 1.0)


@pytest.mark.parametrize("n", [2, 3, 5])
@pytest.mark.parametrize("down,up", [(1e6, 3e6), (3e6, 1e6)])
def test_all_reduce_rate_limited_by_the_slower_direction(n, down, up):
    # every peer sends and returns 2*(n-1)/n of the vector per step in each
    # direction, so the narrower of download and upload sets the rate
    s = np.full(n, 1e9)
    P = 2e6
    r = lp.solve(s, np.full(n, down), np.full(n, up), B=1.0, P=P, fix_c=np.ones(n))
    assert np.isclose(r["xi"], n * min(down, up) / (2 * (n - 1) * P), rtol=1e-6)


@pytest.mark.parametrize("n", [2, 3, 4, 6])
def test_relaxed_rate_with_spare_compute(n):
    s = np.full(n, 1e12)
    b = np.full(n, 1e6)
    P = 2e6
    r = lp.solve(s, b, b, B=1.0, P=P)
    assert np.isclose(r["xi"], 2 * 1e6 / P, rtol=1e-6)
    assert lp.violation(r, s, b, b, 1.0, P) < 1e-7


@pytest.mark.parametrize("seed", range(6))
def test_relaxation_bounds_binary_choices(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 5))
    s = rng.uniform(0, 200, n)
    s[rng.integers(0, n)] = 0.0               # an auxiliary peer without a GPU
    d = rng.uniform(10, 1000, n) * 1e5
    u = rng.uniform(10, 1000, n) * 1e5
    B, P = 1024.0, 1e7
    relaxed = lp.solve(s, d, u, B, P)
    best = 0.0
    for cb in itertools.product([0.0, 1.0], repeat=n):
        r = lp.solve(s, d, u, B, P, fix_c=np.array(cb))
        if r["xi"] is not None:
            best = max(best, r["xi"])
    assert relaxed["xi"] >= best * (1 - 1e-9)
    assert lp.violation(relaxed, s, d, u, B, P) < 1e-7


def test_regional_limits_and_non_aggregators():
    rng = np.random.default_rng(11)
    n = 5
    s = rng.uniform(50, 100, n)
    d = rng.uniform(100, 1000, n) * 1e5
    u = rng.uniform(100, 1000, n) * 1e5
    t = np.full((n, n), np.inf)
    t[0, 1] = t[1, 0] = 1e5
    agg = np.array([True, True, False, True, True])
    r = lp.solve(s, d, u, 2048.0, 5e6, t=t, can_aggregate=agg)
    assert lp.violation(r, s, d, u, 2048.0, 5e6, t=t, can_aggregate=agg) < 1e-7
    assert r["frac"][2] == 0.0 and np.isclose(r["frac"].sum(), 1.0)
    free = lp.solve(s, d, u, 2048.0, 5e6)
    assert r["xi"] <= free["xi"] * (1 + 1e-9)
