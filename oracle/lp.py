"""Load-balancing LP of Appendix B: TEST INFRASTRUCTURE ONLY (oracle).

The problem (Eq. main_problem_appendix_relaxed), written out literally over
the variables a_ij (throughput sender i -> reducer j), g_ij (throughput
reducer i -> receiver j), c_i in [0, 1] (peer i computes gradients) and the
surrogate xi (steps per second):

    max xi
    s.t. xi <= sum_i s_i c_i / B
         xi <= sum_j g_ji / P                           for every i
         g_ij <= a_ki + (1 - c_k) d_i                   for every i, j, k
         sum_{j != i} (a_ji + g_ji) <= d_i              for every i
         sum_{j != i} (a_ij + g_ij) <= u_i              for every i
         a_ij + g_ij <= t_ij                            for every i, j (finite t)
         a, g >= 0,  0 <= c <= 1

and solved with scipy.optimize.linprog (HiGHS), a library routine.  Shares
(the same appendix, the "fraction" equation): reducer i aggregates a share
proportional to min_j g_ij.  Reading: the minimum runs over receivers j != i
(a reducer's transfer to itself is free and unconstrained by the network).
Peers that cannot compute have s_i = 0; peers that cannot aggregate have
a_ji = g_ij = 0 for every j (the appendix's last paragraph excludes them from
the aggregation terms).
"""

from __future__ import annotations

import numpy as np


def _idx(n):
    a = lambda i, j: i * n + j
    g = lambda i, j: n * n + i * n + j
    c = lambda i: 2 * n * n + i
    xi = 2 * n * n + n
    return a, g, c, xi, 2 * n * n + n + 1


def solve(s, d, u, B, P, t=None, can_aggregate=None, fix_c=None, reduced=False):
    """Solve the relaxed LP.  Returns dict(xi, a, g, c, frac, status).

    fix_c: optional array; where not NaN, c_i is fixed to that value.

    reduced: replace the n^3 aggregation rows g_ij <= a_ki + (1 - c_k) d_i by
    the 2n^2 rows  g_ij <= h_i  and  h_i <= a_ki + (1 - c_k) d_i  with one
    more variable h_i per peer (its aggregation rate).  The two programs have
    the same feasible set in (a, g, c, xi): h_i = max_j g_ij turns a point of
    the first into one of the second, and the second's rows chain into the
    first's.  Only the literal program is the oracle's definition; the
    reduced one exists because HiGHS needs minutes on the literal one past
    ~40 peers, and it is pinned against the literal one in the tests.

    Rates are handed to the solver in whole vectors per second (bandwidths
    divided by P, and P = 1): the same program in other units.  Left in
    parameters per second, the 1/P coefficients sit nine orders of magnitude
    below the bandwidths and HiGHS stops within its tolerances but measurably
    short of the optimum."""
    import scipy.optimize as so
    import scipy.sparse as sp

    s, d, u = (np.asarray(v, dtype=np.float64) for v in (s, d, u))
    n = s.size
    d, u = d / P, u / P
    if t is not None:
        t = np.asarray(t, dtype=np.float64) / P
    Pu = P
    P = 1.0
    a, g, c, xi, nv = _idx(n)
    h0 = nv
    h = lambda i: h0 + i
    if reduced:
        nv += n
    rows, cols, vals, rhs = [], [], [], []
    r = 0

    def add(entries, b):
        nonlocal r
        for col, v in entries:
            rows.append(r)
            cols.append(col)
            vals.append(v)
        rhs.append(b)
        r += 1

    add([(xi, 1.0)] + [(c(i), -s[i] / B) for i in range(n)], 0.0)
    for i in range(n):
        add([(xi, 1.0)] + [(g(j, i), -1.0 / P) for j in range(n)], 0.0)
    if reduced:
        for i in range(n):
            for j in range(n):
                add([(g(i, j), 1.0), (h(i), -1.0)], 0.0)
            for k in range(n):
                add([(h(i), 1.0), (a(k, i), -1.0), (c(k), d[i])], d[i])
    else:
        for i in range(n):
            for j in range(n):
                for k in range(n):
                    add([(g(i, j), 1.0), (a(k, i), -1.0), (c(k), d[i])], d[i])
    for i in range(n):
        add([(a(j, i), 1.0) for j in range(n) if j != i] + [(g(j, i), 1.0) for j in range(n) if j != i], d[i])
        add([(a(i, j), 1.0) for j in range(n) if j != i] + [(g(i, j), 1.0) for j in range(n) if j != i], u[i])
    if t is not None:
        t = np.asarray(t, dtype=np.float64)
        for i in range(n):
            for j in range(n):
                if np.isfinite(t[i, j]):
                    add([(a(i, j), 1.0), (g(i, j), 1.0)], t[i, j])
    A = sp.csr_matrix((vals, (rows, cols)), shape=(r, nv))
    bounds = [(0, None)] * (2 * n * n) + [(0, 1)] * n + [(None, None)] + [(0, None)] * (n if reduced else 0)
    if can_aggregate is not None:
        for i in range(n):
            if not can_aggregate[i]:
                for j in range(n):
                    bounds[a(j, i)] = (0, 0)
                    bounds[g(i, j)] = (0, 0)
    if fix_c is not None:
        for i in range(n):
            if not np.isnan(fix_c[i]):
                bounds[c(i)] = (fix_c[i], fix_c[i])
    obj = np.zeros(nv)
    obj[xi] = -1.0
    res = so.linprog(obj, A_ub=A, b_ub=np.array(rhs), bounds=bounds, method="highs")
    if res.status != 0:
        return dict(status=res.status, xi=None)
    x = res.x
    A_ = x[:n * n].reshape(n, n) * Pu
    G = x[n * n:2 * n * n].reshape(n, n) * Pu
    C = x[2 * n * n:2 * n * n + n]
    return dict(status=0, xi=float(x[xi]), a=A_, g=G, c=C, frac=shares(G))


def shares(G):
    """Aggregation shares from the return rates: frac_i = min_{j != i} g_ij,
    normalised to sum to 1 (a single peer takes everything)."""
    G = np.asarray(G, dtype=np.float64)
    n = G.shape[0]
    if n == 1:
        return np.ones(1)
    eff = np.array([min(G[i, j] for j in range(n) if j != i) for i in range(n)])
    eff = np.maximum(eff, 0.0)
    tot = eff.sum()
    return eff / tot if tot > 0 else np.full(n, 1.0 / n)


def violation(sol, s, d, u, B, P, t=None, can_aggregate=None):
    """Largest violation of the relaxed LP's constraints by a solution (with
    the n^3 constraints written out), relative to the data's scale."""
    s, d, u = (np.asarray(v, dtype=np.float64) for v in (s, d, u))
    A, G, C, xi = sol["a"], sol["g"], sol["c"], sol["xi"]
    n = s.size
    scale = max(d.max(), u.max(), 1.0)
    xs = max(abs(xi), 1e-300)
    # rate constraints relative to xi, bandwidth constraints relative to the
    # largest bandwidth, c bounds absolute
    v = [(xi - (s * C).sum() / B) / xs * scale, -A.min(), -G.min(), -C.min() * scale,
         (C.max() - 1.0) * scale]
    for i in range(n):
        v.append((xi - G[:, i].sum() / P) / xs * scale)
        v.append(sum(A[j, i] + G[j, i] for j in range(n) if j != i) - d[i])
        v.append(sum(A[i, j] + G[i, j] for j in range(n) if j != i) - u[i])
        for j in range(n):
            for k in range(n):
                v.append(G[i, j] - A[k, i] - (1.0 - C[k]) * d[i])
            if t is not None and np.isfinite(t[i, j]):
                v.append(A[i, j] + G[i, j] - t[i, j])
    if can_aggregate is not None:
        for i in range(n):
            if not can_aggregate[i]:
                v.append(np.abs(A[:, i]).max())
                v.append(np.abs(G[i, :]).max())
    worst = max(v)
    return max(worst, 0.0) / scale
