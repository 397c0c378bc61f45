// Load balancer of the averaging round (Appendix B): the relaxed linear
// program that assigns every peer a share of the gradient vector to
// aggregate, solved on the host by a deterministic dense simplex.
//
// The appendix's program (Eq. main_problem_appendix_relaxed) has n^3
// aggregation constraints  g_ij <= a_ki + (1 - c_k) d_i.  They are replaced
// here by an exactly equivalent O(n^2) set with one extra variable per
// reducer, its aggregation rate h_i:
//     g_ij <= h_i            for every j
//     h_i <= a_ki + (1 - c_k) d_i   for every k
// (any feasible point of the original gives one of this system with
// h_i = max_j g_ij, and this system implies the original), so the optimum
// and the feasible set in (a, g, c, xi) are unchanged.
//
// Rates are solved in units of whole vectors per second (bandwidths divided
// by P) so that every coefficient is of the order of the answer.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <vector>

#include "../../include/dedloc.h"

namespace {

struct Tableau {
    int m = 0, nvar = 0;          // rows (constraints), columns (variables + slacks)
    std::vector<double> t;        // (m + 1) x nvar row-major; the last row holds the reduced costs
    std::vector<double> b;        // m + 1 right-hand sides (b[m]: the objective's)
    std::vector<int> basis;       // basic variable of each row
    double &at(int r, int c) { return t[(size_t)r * nvar + c]; }
};

// Maximise obj . x subject to A x <= b (b >= 0), x >= 0, starting from the
// slack basis.  Dantzig's entering rule, switching to Bland's rule (smallest
// index) after a run of degenerate pivots so that the method terminates.
// The tableau stays sparse: a pivot touches only the rows where the entering
// column is nonzero, and in them only the pivot row's nonzero columns.
int simplex(Tableau &T, int max_iter, double eps) {
    const int m = T.m, nv = T.nvar;
    std::vector<double> col(m + 1);  // the entering column, gathered
    std::vector<int> nz;             // nonzero columns of the pivot row
    nz.reserve(nv);
    int degenerate = 0;
    for (int it = 0; it < max_iter; it++) {
        const bool bland = degenerate > 50;
        int e = -1;
        double best = -eps;
        const double *cost = &T.t[(size_t)m * nv];
        for (int j = 0; j < nv; j++) {
            const double rc = cost[j];
            if (rc < -eps) {
                if (bland) {
                    e = j;
                    break;
                }
                if (rc < best) {
                    best = rc;
                    e = j;
                }
            }
        }
        if (e < 0) return 0;  // optimal
        const double *ce = &T.t[e];
        for (int r = 0; r <= m; r++) {
            if (r + 16 <= m) __builtin_prefetch(ce + (size_t)(r + 16) * nv);
            col[r] = ce[(size_t)r * nv];
        }
        int p = -1;
        double ratio = 0.0;
        for (int r = 0; r < m; r++) {
            const double a = col[r];
            if (a > eps) {
                const double q = T.b[r] / a;
                if (p < 0 || q < ratio - 1e-15 || (q <= ratio + 1e-15 && T.basis[r] < T.basis[p])) {
                    p = r;
                    ratio = q;
                }
            }
        }
        if (p < 0) return 1;  // unbounded
        degenerate = ratio <= eps ? degenerate + 1 : 0;
        const double piv = col[p];
        double *prow = &T.t[(size_t)p * nv];
        nz.clear();
        for (int c = 0; c < nv; c++)
            if (prow[c] != 0.0) {
                prow[c] /= piv;
                nz.push_back(c);
            }
        prow[e] = 1.0;
        T.b[p] /= piv;
        for (int r = 0; r <= m; r++) {
            const double f = col[r];
            if (r == p || f == 0.0) continue;
            double *row = &T.t[(size_t)r * nv];
            for (const int c : nz) row[c] -= f * prow[c];
            row[e] = 0.0;
            T.b[r] -= f * T.b[p];
        }
        T.basis[p] = e;
    }
    return 2;  // iteration limit
}

}  // namespace

extern "C" int dedloc_balance(const dedloc_balance_problem *pr, double *xi_out, double *c_out,
                              double *frac_out, uint64_t *weights_out, double *a_out, double *g_out) {
    if (!pr || !pr->s || !pr->d || !pr->u || !xi_out || !c_out || !frac_out) return DEDLOC_ERR_INVALID_ARG;
    const int n = (int)pr->n;
    if (n < 1 || n > DEDLOC_BALANCE_MAX_PEERS || !(pr->B > 0) || !(pr->P > 0)) return DEDLOC_ERR_INVALID_ARG;
    for (int i = 0; i < n; i++)
        if (!(pr->s[i] >= 0) || !(pr->d[i] >= 0) || !(pr->u[i] >= 0)) return DEDLOC_ERR_INVALID_ARG;
    const double P = pr->P;
    auto agg = [&](int i) { return !pr->can_aggregate || pr->can_aggregate[i]; };
    // variable indices
    std::vector<int> va(n * n, -1), vg(n * n, -1), vc(n), vh(n);
    int nv = 0;
    for (int i = 0; i < n; i++)
        for (int j = 0; j < n; j++)
            if (agg(j)) va[i * n + j] = nv++;  // a_ij: sender i -> reducer j
    for (int i = 0; i < n; i++)
        for (int j = 0; j < n; j++)
            if (agg(i)) vg[i * n + j] = nv++;  // g_ij: reducer i -> receiver j
    for (int i = 0; i < n; i++) vc[i] = nv++;
    for (int i = 0; i < n; i++) vh[i] = nv++;
    const int vxi = nv++;
    // rows
    struct Row { std::vector<std::pair<int, double>> e; double b; };
    std::vector<Row> rows;
    {
        Row r;
        r.e.push_back({vxi, 1.0});
        for (int i = 0; i < n; i++) r.e.push_back({vc[i], -pr->s[i] / pr->B});
        r.b = 0.0;
        rows.push_back(r);
    }
    for (int i = 0; i < n; i++) {  // xi <= sum_j g_ji / P  (rates already in vectors/s)
        Row r;
        r.e.push_back({vxi, 1.0});
        for (int j = 0; j < n; j++)
            if (vg[j * n + i] >= 0) r.e.push_back({vg[j * n + i], -1.0});
        r.b = 0.0;
        rows.push_back(r);
    }
    for (int i = 0; i < n; i++) {
        if (!agg(i)) continue;
        for (int j = 0; j < n; j++) rows.push_back(Row{{{vg[i * n + j], 1.0}, {vh[i], -1.0}}, 0.0});
        const double di = pr->d[i] / P;
        for (int k = 0; k < n; k++)
            rows.push_back(Row{{{vh[i], 1.0}, {va[k * n + i], -1.0}, {vc[k], di}}, di});
    }
    for (int i = 0; i < n; i++) {
        Row dn, up;
        for (int j = 0; j < n; j++) {
            if (j == i) continue;
            if (va[j * n + i] >= 0) dn.e.push_back({va[j * n + i], 1.0});
            if (vg[j * n + i] >= 0) dn.e.push_back({vg[j * n + i], 1.0});
            if (va[i * n + j] >= 0) up.e.push_back({va[i * n + j], 1.0});
            if (vg[i * n + j] >= 0) up.e.push_back({vg[i * n + j], 1.0});
        }
        dn.b = pr->d[i] / P;
        up.b = pr->u[i] / P;
        rows.push_back(dn);
        rows.push_back(up);
    }
    if (pr->t) {
        for (int i = 0; i < n; i++)
            for (int j = 0; j < n; j++) {
                const double tij = pr->t[i * n + j];
                if (!isfinite(tij)) continue;
                if (tij < 0) return DEDLOC_ERR_INVALID_ARG;
                Row r;
                if (va[i * n + j] >= 0) r.e.push_back({va[i * n + j], 1.0});
                if (vg[i * n + j] >= 0) r.e.push_back({vg[i * n + j], 1.0});
                r.b = tij / P;
                if (!r.e.empty()) rows.push_back(r);
            }
    }
    for (int i = 0; i < n; i++) rows.push_back(Row{{{vc[i], 1.0}}, 1.0});

    Tableau T;
    T.m = (int)rows.size();
    T.nvar = nv + T.m;
    T.t.assign((size_t)(T.m + 1) * T.nvar, 0.0);
    T.b.assign(T.m + 1, 0.0);
    T.basis.resize(T.m);
    for (int r = 0; r < T.m; r++) {
        for (auto &e : rows[r].e) T.at(r, e.first) += e.second;
        T.at(r, nv + r) = 1.0;
        T.b[r] = rows[r].b;
        T.basis[r] = nv + r;
    }
    T.at(T.m, vxi) = -1.0;  // maximise xi
    const int rc = simplex(T, 200000, 1e-12);
    if (rc != 0) return DEDLOC_ERR_INVALID_ARG;

    std::vector<double> x(nv, 0.0);
    for (int r = 0; r < T.m; r++)
        if (T.basis[r] < nv) x[T.basis[r]] = T.b[r];
    *xi_out = x[vxi];
    for (int i = 0; i < n; i++) c_out[i] = x[vc[i]];
    std::vector<double> eff(n, 0.0);
    double tot = 0.0;
    for (int i = 0; i < n; i++) {
        if (!agg(i)) continue;
        double mn = INFINITY;
        for (int j = 0; j < n; j++)
            if (j != i && x[vg[i * n + j]] < mn) mn = x[vg[i * n + j]];
        if (n == 1) mn = 1.0;
        eff[i] = mn > 0 ? mn : 0.0;
        tot += eff[i];
    }
    for (int i = 0; i < n; i++) frac_out[i] = tot > 0 ? eff[i] / tot : (agg(i) ? 1.0 : 0.0);
    if (tot <= 0) {  // degenerate: equal shares among aggregators
        int na = 0;
        for (int i = 0; i < n; i++) na += agg(i);
        for (int i = 0; i < n; i++) frac_out[i] = agg(i) && na ? 1.0 / na : 0.0;
    }
    if (weights_out)
        for (int i = 0; i < n; i++) weights_out[i] = (uint64_t)llround(frac_out[i] * (double)(1u << 24));
    if (a_out)
        for (int i = 0; i < n * n; i++) a_out[i] = va[i] >= 0 ? x[va[i]] * P : 0.0;
    if (g_out)
        for (int i = 0; i < n * n; i++) g_out[i] = vg[i] >= 0 ? x[vg[i]] * P : 0.0;
    return DEDLOC_OK;
}
