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
* the returned solution satisfies every constraint, and its shares sum to 1;
* Section 3.2's special cases, with the compute indicators fixed to the
  binary choice the relaxation stands for (closed forms derived by hand):
  a parameter server (one peer with no compute and bandwidth for everyone)
  takes the whole aggregation and every worker then runs at its own
  bandwidth, xi = b/P; BytePS-style summation peers (no compute, the
  workers' bandwidth) raise 8 workers from the all-reduce rate 4/7*b/P to
  12/19*b/P and necessarily aggregate;
* the O(n^2) reformulation used for large collaborations has the literal
  program's optimum."""

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


@pytest.mark.parametrize("n", [2, 3, 4, 8])
def test_parameter_server(n):
    """Section 3.2: one peer with a very high bandwidth and no compute turns
    the collaboration into a parameter server.  Workers (c = 1) must each send
    their gradient to every aggregator at its rate, so worker k's upload
    carries h_PS + sum_{i != k} h_i + n h_k <= b while every peer receives
    h_PS + sum_i h_i; summed over the workers, xi*P <= b - (n-1)/n * H with H
    the workers' total aggregation: the optimum has H = 0, the server takes
    the whole vector (share 1) and xi = b/P, each worker's link saturated."""
    b, P = 1e6, 1e6
    s = np.array([1e9] * n + [0.0])
    bw = np.array([b] * n + [2 * n * b])
    r = lp.solve(s, bw, bw, B=1.0, P=P, fix_c=np.array([1.0] * n + [0.0]))
    assert np.isclose(r["xi"], b / P, rtol=1e-9)
    assert np.allclose(r["frac"], [0.0] * n + [1.0], atol=1e-9)
    if n > 2:  # better than the workers' own all-reduce
        assert r["xi"] > n * b / (2 * (n - 1) * P) * 1.01


def test_byteps_summation_peers():
    """Section 3.2: peers with the workers' bandwidth and no compute act as
    BytePS summation servers.  8 workers (c = 1) and 8 such peers (c = 0), all
    with bandwidth b; in a symmetric optimum (which exists: the program is
    convex and symmetric) a worker aggregates h_w and a summation peer h_a,
    and the binding constraints are the worker's upload, 22 h_w + 8 h_a <= b,
    and the summation peer's download, 8 h_w + 15 h_a <= b: h_w = b/38,
    h_a = b/19, xi*P = 8 (h_w + h_a) = 12/19 b, against 4/7 b for the
    workers' all-reduce alone.  Without the summation peers aggregating,
    every worker would also have to send the average to them, capping xi*P
    at 8/22 b: so they do aggregate."""
    b, P = 1e6, 1e6
    s = np.array([1e9] * 8 + [0.0] * 8)
    bw = np.full(16, b)
    r = lp.solve(s, bw, bw, B=1.0, P=P, fix_c=np.array([1.0] * 8 + [0.0] * 8))
    assert np.isclose(r["xi"], 12.0 / 19.0 * b / P, rtol=1e-9)
    assert r["xi"] > 4.0 / 7.0 * b / P
    assert r["frac"][8:].sum() > 0.0


@pytest.mark.parametrize("n", [1, 2, 3, 5, 8, 12])
@pytest.mark.parametrize("variant", ["plain", "fixed", "regional", "no_agg"])
def test_reduced_form_has_the_literal_optimum(n, variant):
    rng = np.random.default_rng(100 * n + len(variant))
    s = rng.uniform(1, 200, n)
    d = rng.uniform(10, 1000, n) * 2.5e4
    u = rng.uniform(10, 1000, n) * 2.5e4
    kw = {}
    if variant == "fixed":
        kw["fix_c"] = np.where(rng.uniform(size=n) < 0.5, 1.0, np.nan)
    if variant == "regional":
        t = np.full((n, n), np.inf)
        for _ in range(n):
            i, j = rng.integers(0, n, 2)
            t[i, j] = rng.uniform(1, 50) * 2.5e4
        kw["t"] = t
    if variant == "no_agg":
        kw["can_aggregate"] = rng.uniform(size=n) < 0.7
    lit = lp.solve(s, d, u, 4096.0, 2e7, **kw)
    red = lp.solve(s, d, u, 4096.0, 2e7, reduced=True, **kw)
    assert lit["status"] == 0 and red["status"] == 0
    assert np.isclose(red["xi"], lit["xi"], rtol=1e-9, atol=1e-15)
    assert lp.violation(red, s, d, u, 4096.0, 2e7, t=kw.get("t"), can_aggregate=kw.get("can_aggregate")) < 1e-9
