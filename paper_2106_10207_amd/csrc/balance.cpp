// Load balancer of the averaging round (Appendix B): the relaxed linear
// program that assigns every peer a share of the gradient vector to
// aggregate, solved on the host by a deterministic primal-dual interior-point
// method (the appendix solves it with an interior-point solver too).
//
// The appendix's program (Eq. main_problem_appendix_relaxed) has n^3
// aggregation constraints  g_ij <= a_ki + (1 - c_k) d_i.  They are replaced
// here by an exactly equivalent O(n^2) set with one extra variable per
// reducer, its aggregation rate h_i:
//     g_ij <= h_i            for every j
//     h_i <= a_ki + (1 - c_k) d_i   for every k
// (any feasible point of the original gives one of this system with
// h_i = max_j g_ij, and this system implies the original), so the optimum
// and the feasible set in (a, g, c, xi) are unchanged.  A reducer's transfer
// to itself costs no bandwidth, so a_ii is left out (the constraint with
// k = i holds for a large enough a_ii) unless a finite t_ii limits it.
//
// Rates are solved in units of whole vectors per second (bandwidths divided
// by P) so that every coefficient is of the order of the answer.
//
// Newton systems.  Every variable a_pq (sender p -> reducer q) and g_pq
// (reducer p -> receiver q) appears in at most three "local" rows
// (h_q <= a_pq + (1 - c_p) d_q, g_pq <= h_p, a_pq + g_pq <= t_pq) that touch
// no other a or g, plus the "coupling" rows: peer downloads, uploads and
// receive rates, and the compute row.  Each pair (p, q) is a block of at most
// two variables and three rows; eliminating the blocks leaves a dense
// symmetric quasi-definite system over the coupling unknowns (h, c, xi and
// the multipliers of the 3n + 1 coupling rows, about 5n in all), factored
// once per iteration by LDL^T.  Everything runs in a fixed order, so equal
// inputs give equal outputs bit for bit.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "../../include/dedloc.h"

namespace {

const double kInf = INFINITY;

// min cost.x  s.t.  A x <= b,  0 <= x <= ub (ub may be infinite).
struct Lp {
    int nv = 0, nr = 0;
    std::vector<double> cost, ub, b;
    std::vector<int> rp, rc;      // rows: CSR
    std::vector<double> rv;
    std::vector<int> cp, cr;      // columns: CSC
    std::vector<double> cv;
    // dense system: variable j at gvar[j] (or -1), coupling row r at grow[r]
    // (or -1: a local row); positions [0, ngv) hold variables, [ngv, ng) rows
    std::vector<int> gvar, grow;
    int ngv = 0, ng = 0;
    struct Block {
        int var[2], nvar;
        int row[3], nrow;
    };
    std::vector<Block> blocks;
    std::vector<int> local_rows;  // every local row (each in exactly one block)
};

struct LpBuilder {
    Lp &lp;
    std::vector<std::vector<std::pair<int, double>>> rows;
    explicit LpBuilder(Lp &l) : lp(l) {}
    int var(double cost, double ub, bool global) {
        lp.cost.push_back(cost);
        lp.ub.push_back(ub);
        lp.gvar.push_back(global ? lp.ngv++ : -1);
        return lp.nv++;
    }
    int row(std::vector<std::pair<int, double>> e, double rhs, bool global) {
        rows.push_back(std::move(e));
        lp.b.push_back(rhs);
        lp.grow.push_back(global ? 1 : -1);
        return lp.nr++;
    }
    void finish() {
        lp.rp.assign(1, 0);
        std::vector<int> cnt(lp.nv, 0);
        for (auto &r : rows) {
            for (auto &e : r) {
                lp.rc.push_back(e.first);
                lp.rv.push_back(e.second);
                cnt[e.first]++;
            }
            lp.rp.push_back((int)lp.rc.size());
        }
        lp.cp.assign(lp.nv + 1, 0);
        for (int j = 0; j < lp.nv; j++) lp.cp[j + 1] = lp.cp[j] + cnt[j];
        lp.cr.assign(lp.rc.size(), 0);
        lp.cv.assign(lp.rc.size(), 0.0);
        std::vector<int> fill(lp.cp.begin(), lp.cp.end() - 1);
        for (int r = 0; r < lp.nr; r++)
            for (int k = lp.rp[r]; k < lp.rp[r + 1]; k++) {
                const int j = lp.rc[k];
                lp.cr[fill[j]] = r;
                lp.cv[fill[j]++] = lp.rv[k];
            }
        lp.ng = lp.ngv;
        for (int r = 0; r < lp.nr; r++) {
            if (lp.grow[r] > 0) lp.grow[r] = lp.ng++;
            else lp.local_rows.push_back(r);
        }
    }
};

// Dense symmetric indefinite L D L^T with Bunch-Kaufman pivoting (1x1 and
// 2x2 diagonal blocks, symmetric interchanges) on the lower triangle, stored
// by columns, in the arrangement of LAPACK's unblocked lower factorisation:
// the interchange of step k is applied to the trailing matrix only and
// recorded in piv[k], and the solve replays the interchanges between the
// columns of L.  The reduced Newton systems are quasi-definite, so any pivot
// order exists in exact arithmetic, but a fixed order loses every digit once
// the interior point nears the optimum (pivots of 1e-11 beside entries of
// 1e11); the pivoting keeps the factorisation backward stable.  No fused
// multiply-add anywhere, so the vector clone computes the same bits.
struct Ldl {
    int n = 0;
    std::vector<double> a;      // A(i, j), i >= j, at a[j * n + i]; L below the pivots after factor()
    std::vector<int> piv, blk;  // interchange of each step; block size at a pivot's first index (0 inside)
    std::vector<double> w0, w1;
    double &at(int i, int j) { return a[(size_t)j * n + i]; }
    double at(int i, int j) const { return a[(size_t)j * n + i]; }
    void reserve() {
        a.assign((size_t)n * n, 0.0);
        w0.assign(n, 0.0);
        w1.assign(n, 0.0);
        piv.assign(n, 0);
        blk.assign(n, 0);
    }
    void interchange(int k, int kk, int kp, int size) {  // rows/columns kk <-> kp of A(k:n, k:n), kk < kp
        for (int i = kp + 1; i < n; i++) std::swap(at(i, kk), at(i, kp));
        for (int j = kk + 1; j < kp; j++) std::swap(at(j, kk), at(kp, j));
        std::swap(at(kk, kk), at(kp, kp));
        if (size == 2) std::swap(at(k + 1, k), at(kp, k));
    }
    // A(i, j) -= w0_i L(j, k) (+ w1_i L(j, k+1)) for from <= j <= i, with w the
    // pivot columns before scaling
    __attribute__((target_clones("avx2", "default"))) void update(int from, int k, int size) {
        const double *l0 = &a[(size_t)k * n], *l1 = &a[(size_t)(k + 1) * n];
        const double *x0 = w0.data(), *x1 = w1.data();
        for (int j = from; j < n; j++) {
            double *cj = &a[(size_t)j * n];
            const double v0 = l0[j];
            if (size == 1) {
                if (v0 == 0.0) continue;
                for (int i = j; i < n; i++) cj[i] -= x0[i] * v0;
            } else {
                const double v1 = l1[j];
                for (int i = j; i < n; i++) cj[i] -= x0[i] * v0 + x1[i] * v1;
            }
        }
    }
    void factor() {
        const double alpha = (1.0 + sqrt(17.0)) / 8.0;
        int k = 0;
        while (k < n) {
            const double akk = fabs(at(k, k));
            int imax = k;
            double colmax = 0.0;
            for (int i = k + 1; i < n; i++)
                if (fabs(at(i, k)) > colmax) {
                    colmax = fabs(at(i, k));
                    imax = i;
                }
            int size = 1, kp = k;
            if (std::max(akk, colmax) == 0.0) {
                at(k, k) = 1e-300;  // an empty column: its unknown is free
            } else if (akk < alpha * colmax) {
                double rowmax = 0.0;
                for (int j = k; j < imax; j++) rowmax = std::max(rowmax, fabs(at(imax, j)));
                for (int i = imax + 1; i < n; i++) rowmax = std::max(rowmax, fabs(at(i, imax)));
                if (akk >= alpha * colmax * (colmax / rowmax)) {
                    kp = k;
                } else if (fabs(at(imax, imax)) >= alpha * rowmax) {
                    kp = imax;
                } else {
                    kp = imax;
                    size = 2;
                }
            }
            const int kk = k + size - 1;
            if (kp != kk) interchange(k, kk, kp, size);
            blk[k] = size;
            if (size == 2) blk[k + 1] = 0;
            piv[k] = kp;
            if (size == 1) {
                const double d = at(k, k);
                for (int i = k + 1; i < n; i++) {
                    w0[i] = at(i, k);
                    at(i, k) = w0[i] / d;
                }
                update(k + 1, k, 1);
            } else {
                const double a11 = at(k, k), a21 = at(k + 1, k), a22 = at(k + 1, k + 1);
                const double det = a11 * a22 - a21 * a21;
                for (int i = k + 2; i < n; i++) {
                    const double x0 = at(i, k), x1 = at(i, k + 1);
                    w0[i] = x0;
                    w1[i] = x1;
                    at(i, k) = (x0 * a22 - x1 * a21) / det;
                    at(i, k + 1) = (x1 * a11 - x0 * a21) / det;
                }
                update(k + 2, k, 2);
            }
            k += size;
        }
    }
    void solve(double *b) const {
        int k = 0;
        while (k < n) {
            const double *c0 = &a[(size_t)k * n];
            if (blk[k] == 1) {
                if (piv[k] != k) std::swap(b[k], b[piv[k]]);
                const double bk = b[k];
                for (int i = k + 1; i < n; i++) b[i] -= c0[i] * bk;
                b[k] = bk / c0[k];
                k += 1;
            } else {
                const double *c1 = &a[(size_t)(k + 1) * n];
                if (piv[k] != k + 1) std::swap(b[k + 1], b[piv[k]]);
                const double b0 = b[k], b1 = b[k + 1];
                for (int i = k + 2; i < n; i++) b[i] -= c0[i] * b0 + c1[i] * b1;
                const double a11 = c0[k], a21 = c0[k + 1], a22 = c1[k + 1];
                const double det = a11 * a22 - a21 * a21;
                b[k] = (a22 * b0 - a21 * b1) / det;
                b[k + 1] = (a11 * b1 - a21 * b0) / det;
                k += 2;
            }
        }
        k = n - 1;
        while (k >= 0) {
            if (blk[k] == 1) {
                const double *c0 = &a[(size_t)k * n];
                double sum = b[k];
                for (int i = k + 1; i < n; i++) sum -= c0[i] * b[i];
                b[k] = sum;
                if (piv[k] != k) std::swap(b[k], b[piv[k]]);
                k -= 1;
            } else {  // blk[k] == 0: the second index of the 2x2 block starting at k - 1
                const double *c0 = &a[(size_t)(k - 1) * n], *c1 = &a[(size_t)k * n];
                double s1 = b[k], s0 = b[k - 1];
                for (int i = k + 1; i < n; i++) {
                    s1 -= c1[i] * b[i];
                    s0 -= c0[i] * b[i];
                }
                b[k] = s1;
                b[k - 1] = s0;
                if (piv[k - 1] != k) std::swap(b[k], b[piv[k - 1]]);
                k -= 2;
            }
        }
    }
};

// The Newton system  [Tinv  A^T; A  -E] [dx; dy] = [rd; rp]  (Tinv, E positive
// diagonals).  The a and g variables are eliminated as in the normal
// equations (dx_s = Theta_s (rd_s - A_s^T dy)), which leaves
//     [N       -A_D   ] [dy  ]   [-rp + A_s Theta_s rd_s]
//     [-A_D^T  -Tinv_D] [dx_D] = [-rd_D                ],   N = A_s Theta_s A_s^T + E,
// over every row and the dense variables D = (h, c, xi).  N couples a
// block's local rows only with each other and with the coupling rows, so
// each block's (at most 3x3, positive definite) part is eliminated, leaving
// a dense symmetric system over the coupling rows and D.  Iterative
// refinement on the unreduced system cleans up the rounding.
class Kkt {
    static constexpr int kMaxG = 6;  // dense unknowns one block touches (6 in this program)

  public:
    explicit Kkt(const Lp &lp) : lp_(lp) {
        pos_row_.assign(lp.nr, -1);
        pos_var_.assign(lp.nv, -1);
        int g = 0;
        for (int r = 0; r < lp.nr; r++)
            if (lp.grow[r] >= 0) pos_row_[r] = g++;
        for (int j = 0; j < lp.nv; j++)
            if (lp.gvar[j] >= 0) pos_var_[j] = g++;
        ng_ = g;
        ldl_.n = ng_;
        ldl_.reserve();
        theta_.assign(lp.nv, 0.0);
        loc_.resize(lp.blocks.size());
        coef_.resize(lp.blocks.size());
        for (size_t bi = 0; bi < lp.blocks.size(); bi++) setup(lp.blocks[bi], loc_[bi], coef_[bi]);
    }

    // False when a block touched more dense unknowns than kMaxG (the
    // program's structure allows 6); the system is then not set up.
    bool ok() const { return ok_; }

    void factor(const std::vector<double> &tinv, const std::vector<double> &e) {
        tinv_ = &tinv;
        e_ = &e;
        for (int j = 0; j < lp_.nv; j++) theta_[j] = 1.0 / tinv[j];
        std::vector<double> &S = ldl_.a;
        std::fill(S.begin(), S.end(), 0.0);
        const int ng = ng_;
        auto add = [&S, ng](int i, int j, double v) {
            if (i < j) std::swap(i, j);
            S[(size_t)j * ng + i] += v;
        };
        // coupling rows: E, and A_C Theta_s A_C^T over the sparse variables
        for (int r = 0; r < lp_.nr; r++)
            if (pos_row_[r] >= 0) add(pos_row_[r], pos_row_[r], e[r]);
        for (int j = 0; j < lp_.nv; j++) {
            if (pos_var_[j] >= 0) continue;
            for (int k = lp_.cp[j]; k < lp_.cp[j + 1]; k++) {
                const int pi = pos_row_[lp_.cr[k]];
                if (pi < 0) continue;
                for (int q = lp_.cp[j]; q <= k; q++) {
                    const int pj = pos_row_[lp_.cr[q]];
                    if (pj >= 0) add(pi, pj, theta_[j] * lp_.cv[k] * lp_.cv[q]);
                }
            }
        }
        // coupling rows x D and D x D
        for (int j = 0; j < lp_.nv; j++) {
            const int pj = pos_var_[j];
            if (pj < 0) continue;
            add(pj, pj, -tinv[j]);
            for (int k = lp_.cp[j]; k < lp_.cp[j + 1]; k++) {
                const int pr = pos_row_[lp_.cr[k]];
                if (pr >= 0) add(pr, pj, -lp_.cv[k]);
            }
        }
        // eliminate every block's local rows: S -= W^T K^-1 W
        for (size_t bi = 0; bi < lp_.blocks.size(); bi++) {
            const Lp::Block &B = lp_.blocks[bi];
            Local &L = loc_[bi];
            const Coef &C = coef_[bi];
            const double th[2] = {theta_[B.var[0]], B.nvar > 1 ? theta_[B.var[1]] : 0.0};
            double K[3][3] = {{0}};
            for (int t = 0; t < B.nrow; t++) {
                K[t][t] = e[B.row[t]];
                for (int u = 0; u <= t; u++)
                    for (int v = 0; v < B.nvar; v++) K[t][u] += th[v] * C.arv[t][v] * C.arv[u][v];
                for (int g = 0; g < L.ng; g++) L.w[t][g] = C.cst[t][g] + th[0] * C.cv[t][g][0] + th[1] * C.cv[t][g][1];
            }
            L.factor(K, B.nrow);
            double kw[3][kMaxG];  // K^-1 W
            for (int g = 0; g < L.ng; g++) {
                double col[3];
                for (int t = 0; t < B.nrow; t++) col[t] = L.w[t][g];
                L.solve(col, B.nrow);
                for (int t = 0; t < B.nrow; t++) kw[t][g] = col[t];
            }
            for (int g = 0; g < L.ng; g++)
                for (int h = 0; h < L.ng; h++) {
                    if (L.pos[h] > L.pos[g]) continue;  // lower triangle only
                    double v = 0.0;
                    for (int t = 0; t < B.nrow; t++) v += L.w[t][g] * kw[t][h];
                    add(L.pos[g], L.pos[h], -v);
                }
        }
        ldl_.factor();
    }

    void solve(const std::vector<double> &rd, const std::vector<double> &rp, std::vector<double> &dx,
               std::vector<double> &dy) {
        dx.assign(lp_.nv, 0.0);
        dy.assign(lp_.nr, 0.0);
        once(rd, rp, dx, dy);
        ex_.resize(lp_.nv);
        ey_.resize(lp_.nr);
        cx_.resize(lp_.nv);
        cy_.resize(lp_.nr);
        double rhs = 0.0;
        for (double v : rd) rhs = std::max(rhs, fabs(v));
        for (double v : rp) rhs = std::max(rhs, fabs(v));
        for (int it = 0; it < 4; it++) {
            double worst = 0.0;
            for (int j = 0; j < lp_.nv; j++) {
                double s = (*tinv_)[j] * dx[j];
                for (int k = lp_.cp[j]; k < lp_.cp[j + 1]; k++) s += lp_.cv[k] * dy[lp_.cr[k]];
                cx_[j] = rd[j] - s;
                worst = std::max(worst, fabs(cx_[j]) * std::min(theta_[j], 1.0));
            }
            for (int r = 0; r < lp_.nr; r++) {
                double s = -(*e_)[r] * dy[r];
                for (int k = lp_.rp[r]; k < lp_.rp[r + 1]; k++) s += lp_.rv[k] * dx[lp_.rc[k]];
                cy_[r] = rp[r] - s;
                worst = std::max(worst, fabs(cy_[r]));
            }
            if (worst <= 1e-15 * (1.0 + rhs)) break;
            once(cx_, cy_, ex_, ey_);
            for (int j = 0; j < lp_.nv; j++) dx[j] += ex_[j];
            for (int r = 0; r < lp_.nr; r++) dy[r] += ey_[r];
        }
    }

  private:
    // A block's local rows, in two records: what every solve reads (the
    // dense unknowns they couple to, W = cst + theta_0 cv_0 + theta_1 cv_1 for
    // the current theta, and the factor of their N block) and what only the
    // factorisation reads (their coefficients on the block's variables, and
    // W's parts: -A_D entries, and through a block variable the coupling rows
    // it is in).  Kept apart, the solves stream a third of the bytes.
    struct Coef {
        double arv[3][2];
        double cst[3][kMaxG], cv[3][kMaxG][2];
    };
    struct Local {
        int ng = 0;
        int pos[kMaxG];
        double w[3][kMaxG];
        double l[3][3], dg[3];
        void factor(double K[3][3], int m) {
            double dmax = 0.0;
            for (int i = 0; i < m; i++) dmax = std::max(dmax, K[i][i]);
            for (int i = 0; i < m; i++) {
                for (int j = 0; j < i; j++) {
                    double s = K[i][j];
                    for (int k = 0; k < j; k++) s -= l[i][k] * dg[k] * l[j][k];
                    l[i][j] = s / dg[j];
                }
                double s = K[i][i];
                for (int k = 0; k < i; k++) s -= l[i][k] * dg[k] * l[i][k];
                dg[i] = s > 1e-30 * dmax ? s : 1e128;  // degenerate row (active, its variables at bounds): step ~0
            }
        }
        void solve(double *x, int m) const {
            for (int i = 0; i < m; i++)
                for (int k = 0; k < i; k++) x[i] -= l[i][k] * x[k];
            for (int i = 0; i < m; i++) x[i] /= dg[i];
            for (int i = m - 1; i >= 0; i--)
                for (int k = i + 1; k < m; k++) x[i] -= l[k][i] * x[k];
        }
        int slot(int p, Coef &c) {  // -1: more than kMaxG dense unknowns
            for (int g = 0; g < ng; g++)
                if (pos[g] == p) return g;
            if (ng == kMaxG) return -1;
            pos[ng] = p;
            for (int t = 0; t < 3; t++) c.cst[t][ng] = c.cv[t][ng][0] = c.cv[t][ng][1] = 0.0;
            return ng++;
        }
    };

    void setup(const Lp::Block &B, Local &L, Coef &C) {
        L.ng = 0;
        for (int t = 0; t < B.nrow; t++) {
            const int r = B.row[t];
            for (int v = 0; v < 2; v++) C.arv[t][v] = 0.0;
            for (int k = lp_.rp[r]; k < lp_.rp[r + 1]; k++) {
                const int j = lp_.rc[k];
                if (pos_var_[j] >= 0) {
                    const int g = L.slot(pos_var_[j], C);
                    if (g < 0) {
                        ok_ = false;
                        return;
                    }
                    C.cst[t][g] += -lp_.rv[k];  // -A_D
                    continue;
                }
                for (int v = 0; v < B.nvar; v++)
                    if (B.var[v] == j) {
                        C.arv[t][v] = lp_.rv[k];
                        for (int q = lp_.cp[j]; q < lp_.cp[j + 1]; q++) {
                            const int pr = pos_row_[lp_.cr[q]];
                            if (pr < 0) continue;
                            const int g = L.slot(pr, C);
                            if (g < 0) {
                                ok_ = false;
                                return;
                            }
                            C.cv[t][g][v] += lp_.rv[k] * lp_.cv[q];
                        }
                    }
            }
        }
    }

    void once(const std::vector<double> &rd, const std::vector<double> &rp, std::vector<double> &dx,
              std::vector<double> &dy) {
        rr_.resize(lp_.nr);
        u_.assign(ng_, 0.0);
        std::vector<double> &rr = rr_, &u = u_;
        for (int r = 0; r < lp_.nr; r++) {
            double s = -rp[r];
            for (int k = lp_.rp[r]; k < lp_.rp[r + 1]; k++) {
                const int j = lp_.rc[k];
                if (pos_var_[j] < 0) s += lp_.rv[k] * theta_[j] * rd[j];
            }
            rr[r] = s;
            if (pos_row_[r] >= 0) u[pos_row_[r]] = s;
        }
        for (int j = 0; j < lp_.nv; j++)
            if (pos_var_[j] >= 0) u[pos_var_[j]] = -rd[j];
        for (size_t bi = 0; bi < lp_.blocks.size(); bi++) {
            const Lp::Block &B = lp_.blocks[bi];
            const Local &L = loc_[bi];
            double t[3] = {0, 0, 0};
            for (int i = 0; i < B.nrow; i++) t[i] = rr[B.row[i]];
            L.solve(t, B.nrow);
            for (int g = 0; g < L.ng; g++) {
                double v = 0.0;
                for (int i = 0; i < B.nrow; i++) v += L.w[i][g] * t[i];
                u[L.pos[g]] -= v;
            }
        }
        ldl_.solve(u.data());
        for (int r = 0; r < lp_.nr; r++)
            if (pos_row_[r] >= 0) dy[r] = u[pos_row_[r]];
        for (int j = 0; j < lp_.nv; j++)
            if (pos_var_[j] >= 0) dx[j] = u[pos_var_[j]];
        for (size_t bi = 0; bi < lp_.blocks.size(); bi++) {
            const Lp::Block &B = lp_.blocks[bi];
            const Local &L = loc_[bi];
            double t[3] = {0, 0, 0};
            for (int i = 0; i < B.nrow; i++) {
                t[i] = rr[B.row[i]];
                for (int g = 0; g < L.ng; g++) t[i] -= L.w[i][g] * u[L.pos[g]];
            }
            L.solve(t, B.nrow);
            for (int i = 0; i < B.nrow; i++) dy[B.row[i]] = t[i];
        }
        for (int j = 0; j < lp_.nv; j++) {
            if (pos_var_[j] >= 0) continue;
            double s = rd[j];
            for (int k = lp_.cp[j]; k < lp_.cp[j + 1]; k++) s -= lp_.cv[k] * dy[lp_.cr[k]];
            dx[j] = theta_[j] * s;
        }
    }

    const Lp &lp_;
    std::vector<int> pos_row_, pos_var_;
    int ng_ = 0;
    Ldl ldl_;
    std::vector<double> theta_, rr_, u_, ex_, ey_, cx_, cy_;
    std::vector<Local> loc_;
    std::vector<Coef> coef_;
    bool ok_ = true;
    const std::vector<double> *tinv_ = nullptr, *e_ = nullptr;
};

// Largest step in (0, 1] keeping v + alpha * dv >= 0 for every v, scaled by
// `frac`.
double step_to_boundary(const std::vector<double> &v, const std::vector<double> &dv, const std::vector<char> &on,
                        double frac) {
    double a = 1.0;
    for (size_t i = 0; i < v.size(); i++)
        if (on[i] && dv[i] < 0.0) a = std::min(a, -v[i] / dv[i] * frac);
    return a;
}

// Primal-dual interior point (Mehrotra's predictor-corrector) for
//   min c.x  s.t.  A x + w = b, w >= 0,  x >= 0,  x + s = ub (finite ub), s >= 0.
// Returns 0 when converged, 1 otherwise; x holds the last iterate.
int interior_point(const Lp &lp, std::vector<double> &x, int *iterations) {
    const int nv = lp.nv, nr = lp.nr;
    std::vector<char> hasub(nv), allv(nv, 1), allr(nr, 1);
    for (int j = 0; j < nv; j++) hasub[j] = isfinite(lp.ub[j]);
    x.assign(nv, 0.0);
    std::vector<double> z(nv, 1.0), s(nv, 0.0), q(nv, 0.0), w(nr), y(nr, 1.0);
    for (int j = 0; j < nv; j++) {
        x[j] = hasub[j] ? std::min(0.5 * lp.ub[j], 1.0) : 1.0;
        if (hasub[j]) {
            s[j] = lp.ub[j] - x[j];
            q[j] = 1.0;
        }
    }
    double cnorm = 0.0;
    for (int r = 0; r < nr; r++) {
        double ax = 0.0;
        for (int k = lp.rp[r]; k < lp.rp[r + 1]; k++) ax += lp.rv[k] * x[lp.rc[k]];
        w[r] = std::max(lp.b[r] - ax, 1.0);
    }
    for (int j = 0; j < nv; j++) cnorm = std::max(cnorm, fabs(lp.cost[j]));
    const int ncomp = nv + nr + (int)std::count(hasub.begin(), hasub.end(), 1);

    Kkt kkt(lp);
    if (!kkt.ok()) return 1;
    std::vector<double> rp(nr), rd(nv), tinv(nv), e(nr), rhs_d(nv), rhs_p(nr);
    std::vector<double> dx, dy, dz(nv), ds(nv), dq(nv), dw(nr);
    std::vector<double> ax_(nv), ay_(nr), az_(nv), as_(nv), aq_(nv), aw_(nr);  // affine direction
    auto residuals = [&](double &pinf, double &dinf, double &pobj, double &dobj) {
        pinf = dinf = 0.0;
        for (int r = 0; r < nr; r++) {
            double v = w[r] - lp.b[r], mag = 1.0 + fabs(lp.b[r]) + w[r];
            for (int k = lp.rp[r]; k < lp.rp[r + 1]; k++) {
                v += lp.rv[k] * x[lp.rc[k]];
                mag += fabs(lp.rv[k] * x[lp.rc[k]]);
            }
            rp[r] = v;
            // row by row, relative to the magnitudes the row adds up
            pinf = isnan(v) ? NAN : std::max(pinf, fabs(v) / mag);
        }
        pobj = dobj = 0.0;
        for (int j = 0; j < nv; j++) {
            double v = lp.cost[j] - z[j] + (hasub[j] ? q[j] : 0.0);
            for (int k = lp.cp[j]; k < lp.cp[j + 1]; k++) v += lp.cv[k] * y[lp.cr[k]];
            rd[j] = v;
            dinf = isnan(v) ? NAN : std::max(dinf, fabs(v));
            pobj += lp.cost[j] * x[j];
            if (hasub[j]) dobj -= lp.ub[j] * q[j];
        }
        for (int r = 0; r < nr; r++) dobj -= lp.b[r] * y[r];
    };
    // solve for complementarity targets given by rxz, rwy, rsq (per element)
    auto direction = [&](const std::vector<double> &rxz, const std::vector<double> &rwy,
                         const std::vector<double> &rsq, std::vector<double> &Dx, std::vector<double> &Dy,
                         std::vector<double> &Dz, std::vector<double> &Ds, std::vector<double> &Dq,
                         std::vector<double> &Dw) {
        for (int j = 0; j < nv; j++) rhs_d[j] = -rd[j] - rxz[j] / x[j] + (hasub[j] ? rsq[j] / s[j] : 0.0);
        for (int r = 0; r < nr; r++) rhs_p[r] = -rp[r] + rwy[r] / y[r];
        kkt.solve(rhs_d, rhs_p, Dx, Dy);
        for (int j = 0; j < nv; j++) {
            Dz[j] = (-rxz[j] - z[j] * Dx[j]) / x[j];
            if (hasub[j]) {
                Ds[j] = -Dx[j];
                Dq[j] = (-rsq[j] + q[j] * Dx[j]) / s[j];
            } else {
                Ds[j] = Dq[j] = 0.0;
            }
        }
        for (int r = 0; r < nr; r++) Dw[r] = (-rwy[r] - w[r] * Dy[r]) / y[r];
    };
    std::vector<double> rxz(nv), rwy(nr), rsq(nv);
    // the most accurate iterate so far (in case rounding stalls the last
    // digits): accepted if it is within 1e-9 on every measure
    std::vector<double> best;
    double best_err = INFINITY;
    for (int it = 0; it < 200; it++) {
        double pinf, dinf, pobj, dobj;
        residuals(pinf, dinf, pobj, dobj);
        double mu = 0.0;
        for (int j = 0; j < nv; j++) mu += x[j] * z[j] + (hasub[j] ? s[j] * q[j] : 0.0);
        for (int r = 0; r < nr; r++) mu += w[r] * y[r];
        mu /= ncomp;
        const double gap = fabs(pobj - dobj) / std::max(std::max(fabs(pobj), fabs(dobj)), 1e-300);
        if (iterations) *iterations = it;
        if (pinf <= 1e-11 && dinf <= 1e-11 * (1.0 + cnorm) && (gap <= 1e-12 || mu <= 1e-300)) return 0;
        double err = std::max({pinf, dinf / (1.0 + cnorm), gap});
        if (!isfinite(pinf) || !isfinite(dinf) || !isfinite(gap)) err = INFINITY;
        if (!(err < best_err)) {
            if (!(err <= 10.0 * best_err) || !isfinite(err)) break;  // going astray: stop
        } else {
            best_err = err;
            best = x;
        }
        for (int j = 0; j < nv; j++) {
            tinv[j] = z[j] / x[j] + (hasub[j] ? q[j] / s[j] : 0.0);
        }
        for (int r = 0; r < nr; r++) e[r] = w[r] / y[r];
        kkt.factor(tinv, e);
        // predictor (affine scaling)
        for (int j = 0; j < nv; j++) {
            rxz[j] = x[j] * z[j];
            rsq[j] = hasub[j] ? s[j] * q[j] : 0.0;
        }
        for (int r = 0; r < nr; r++) rwy[r] = w[r] * y[r];
        direction(rxz, rwy, rsq, ax_, ay_, az_, as_, aq_, aw_);
        double ap = std::min({step_to_boundary(x, ax_, allv, 1.0), step_to_boundary(s, as_, hasub, 1.0),
                              step_to_boundary(w, aw_, allr, 1.0)});
        double ad = std::min({step_to_boundary(z, az_, allv, 1.0), step_to_boundary(q, aq_, hasub, 1.0),
                              step_to_boundary(y, ay_, allr, 1.0)});
        double mu_aff = 0.0;
        for (int j = 0; j < nv; j++) {
            mu_aff += (x[j] + ap * ax_[j]) * (z[j] + ad * az_[j]);
            if (hasub[j]) mu_aff += (s[j] + ap * as_[j]) * (q[j] + ad * aq_[j]);
        }
        for (int r = 0; r < nr; r++) mu_aff += (w[r] + ap * aw_[r]) * (y[r] + ad * ay_[r]);
        mu_aff /= ncomp;
        const double sigma = std::pow(mu_aff / mu, 3.0);
        // corrector
        for (int j = 0; j < nv; j++) {
            rxz[j] = x[j] * z[j] + ax_[j] * az_[j] - sigma * mu;
            rsq[j] = hasub[j] ? s[j] * q[j] + as_[j] * aq_[j] - sigma * mu : 0.0;
        }
        for (int r = 0; r < nr; r++) rwy[r] = w[r] * y[r] + aw_[r] * ay_[r] - sigma * mu;
        direction(rxz, rwy, rsq, dx, dy, dz, ds, dq, dw);
        bool finite = true;
        for (int j = 0; j < nv && finite; j++) finite = isfinite(dx[j]) && isfinite(dz[j]) && isfinite(dq[j]);
        for (int r = 0; r < nr && finite; r++) finite = isfinite(dy[r]) && isfinite(dw[r]);
        if (!finite) break;  // the Newton system lost its accuracy: keep the best iterate
        const double eta = 0.995;
        ap = std::min({step_to_boundary(x, dx, allv, eta), step_to_boundary(s, ds, hasub, eta),
                       step_to_boundary(w, dw, allr, eta)});
        ad = std::min({step_to_boundary(z, dz, allv, eta), step_to_boundary(q, dq, hasub, eta),
                       step_to_boundary(y, dy, allr, eta)});
        for (int j = 0; j < nv; j++) {
            x[j] += ap * dx[j];
            z[j] += ad * dz[j];
            if (hasub[j]) {
                s[j] += ap * ds[j];
                q[j] += ad * dq[j];
            }
        }
        for (int r = 0; r < nr; r++) {
            w[r] += ap * dw[r];
            y[r] += ad * dy[r];
        }
    }
    if (best_err <= 1e-9) {
        x = best;
        return 0;
    }
    return 1;
}

}  // namespace

extern "C" int dedloc_balance(const dedloc_balance_problem *pr, double *xi_out, double *c_out,
                              double *frac_out, uint64_t *weights_out, double *a_out, double *g_out) {
    if (!pr || !pr->s || !pr->d || !pr->u || !xi_out || !c_out || !frac_out) return DEDLOC_ERR_INVALID_ARG;
    const int n = (int)pr->n;
    if (n < 1 || n > DEDLOC_BALANCE_MAX_PEERS || !(pr->B > 0) || !(pr->P > 0)) return DEDLOC_ERR_INVALID_ARG;
    for (int i = 0; i < n; i++)
        if (!(pr->s[i] >= 0) || !(pr->d[i] >= 0) || !(pr->u[i] >= 0) || !isfinite(pr->s[i]) ||
            !isfinite(pr->d[i]) || !isfinite(pr->u[i]))
            return DEDLOC_ERR_INVALID_ARG;
    if (pr->t)
        for (int i = 0; i < n * n; i++)
            if (pr->t[i] < 0 || isnan(pr->t[i])) return DEDLOC_ERR_INVALID_ARG;
    if (pr->c_fixed)
        for (int i = 0; i < n; i++)
            if (!isnan(pr->c_fixed[i]) && !(pr->c_fixed[i] >= 0.0 && pr->c_fixed[i] <= 1.0))
                return DEDLOC_ERR_INVALID_ARG;
    // a fixed c_k is a constant, not a variable
    auto cfix = [&](int k) { return pr->c_fixed && !isnan(pr->c_fixed[k]); };
    const double P = pr->P;
    auto agg = [&](int i) { return !pr->can_aggregate || pr->can_aggregate[i]; };
    auto tfin = [&](int i, int j) { return pr->t && isfinite(pr->t[i * n + j]); };
    std::vector<double> d(n), u(n);
    double ssum = 0.0;
    for (int i = 0; i < n; i++) {
        d[i] = pr->d[i] / P;
        u[i] = pr->u[i] / P;
        ssum += pr->s[i] / pr->B;
    }

    Lp lp;
    LpBuilder bld(lp);
    const int vxi = bld.var(-1.0, kInf, true);  // maximise xi
    std::vector<int> vc(n, -1), vh(n, -1), va(n * n, -1), vg(n * n, -1);
    for (int k = 0; k < n; k++)
        if (!cfix(k)) vc[k] = bld.var(0.0, 1.0, true);
    // h_i <= d_i + a_ki <= 2 d_i for n >= 2; the bound only keeps the
    // feasible set bounded for n = 1 and is never active otherwise
    for (int i = 0; i < n; i++)
        if (agg(i)) vh[i] = bld.var(0.0, 4.0 * d[i] + 4.0 * ssum + 1.0, true);
    for (int p = 0; p < n; p++)
        for (int q = 0; q < n; q++) {
            if (agg(q) && (p != q || tfin(p, q))) va[p * n + q] = bld.var(0.0, kInf, false);  // a_pq
            if (agg(p)) vg[p * n + q] = bld.var(0.0, kInf, false);                        // g_pq
        }
    {
        std::vector<std::pair<int, double>> e{{vxi, 1.0}};
        double fixed = 0.0;
        for (int k = 0; k < n; k++) {
            if (cfix(k)) fixed += pr->s[k] / pr->B * pr->c_fixed[k];
            else if (pr->s[k] > 0) e.push_back({vc[k], -pr->s[k] / pr->B});
        }
        bld.row(e, fixed, true);
    }
    for (int q = 0; q < n; q++) {  // xi <= sum_p g_pq
        std::vector<std::pair<int, double>> e{{vxi, 1.0}};
        for (int p = 0; p < n; p++)
            if (vg[p * n + q] >= 0) e.push_back({vg[p * n + q], -1.0});
        bld.row(e, 0.0, true);
    }
    for (int i = 0; i < n; i++) {  // download and upload of peer i
        std::vector<std::pair<int, double>> dn, up;
        for (int j = 0; j < n; j++) {
            if (j == i) continue;
            if (va[j * n + i] >= 0) dn.push_back({va[j * n + i], 1.0});
            if (vg[j * n + i] >= 0) dn.push_back({vg[j * n + i], 1.0});
            if (va[i * n + j] >= 0) up.push_back({va[i * n + j], 1.0});
            if (vg[i * n + j] >= 0) up.push_back({vg[i * n + j], 1.0});
        }
        bld.row(dn, d[i], true);
        bld.row(up, u[i], true);
    }
    for (int p = 0; p < n; p++)
        for (int q = 0; q < n; q++) {
            Lp::Block B;
            B.nvar = B.nrow = 0;
            const int a = va[p * n + q], g = vg[p * n + q];
            if (a >= 0) {
                B.var[B.nvar++] = a;
                B.row[B.nrow++] = cfix(p) ? bld.row({{vh[q], 1.0}, {a, -1.0}}, (1.0 - pr->c_fixed[p]) * d[q], false)
                                          : bld.row({{vh[q], 1.0}, {a, -1.0}, {vc[p], d[q]}}, d[q], false);
            }
            if (g >= 0) {
                B.var[B.nvar++] = g;
                B.row[B.nrow++] = bld.row({{g, 1.0}, {vh[p], -1.0}}, 0.0, false);
            }
            if (B.nvar && tfin(p, q)) {
                std::vector<std::pair<int, double>> e;
                if (a >= 0) e.push_back({a, 1.0});
                if (g >= 0) e.push_back({g, 1.0});
                B.row[B.nrow++] = bld.row(e, pr->t[p * n + q] / P, false);
            }
            if (B.nvar) lp.blocks.push_back(B);
        }
    bld.finish();

    std::vector<double> x;
    int iters = 0;
    if (interior_point(lp, x, &iters) != 0) return DEDLOC_ERR_INVALID_ARG;
    for (int j = 0; j < lp.nv; j++) x[j] = std::min(std::max(x[j], 0.0), lp.ub[j]);
    // xi no larger than its own constraints allow at the final point (this
    // moves it by rounding only; with no compute anywhere it is exactly 0)
    {
        double cap = 0.0;
        for (int k = 0; k < n; k++) cap += pr->s[k] / pr->B * (cfix(k) ? pr->c_fixed[k] : x[vc[k]]);
        for (int q = 0; q < n; q++) {
            double in = 0.0;
            for (int p = 0; p < n; p++)
                if (vg[p * n + q] >= 0) in += x[vg[p * n + q]];
            cap = std::min(cap, in);
        }
        x[vxi] = std::min(x[vxi], cap);
    }

    *xi_out = x[vxi];
    for (int i = 0; i < n; i++) c_out[i] = cfix(i) ? pr->c_fixed[i] : x[vc[i]];
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
        for (int p = 0; p < n; p++)
            for (int q = 0; q < n; q++) {
                double v = va[p * n + q] >= 0 ? x[va[p * n + q]] : 0.0;
                if (p == q && agg(q) && va[p * n + q] < 0) {
                    // a reducer's own contribution: free; the smallest value
                    // that satisfies h_q <= a_qq + (1 - c_q) d_q
                    double h = 0.0;
                    for (int j = 0; j < n; j++) h = std::max(h, x[vg[q * n + j]]);
                    v = std::max(0.0, h - (1.0 - c_out[q]) * d[q]);
                }
                a_out[p * n + q] = v * P;
            }
    if (g_out)
        for (int i = 0; i < n * n; i++) g_out[i] = vg[i] >= 0 ? x[vg[i]] * P : 0.0;
    return DEDLOC_OK;
}

// Group size of the group all-reduce (Appendix C): the m minimising
// ceil(log_m n) / (1 - p)^m, as declared in dedloc.h.
extern "C" int dedloc_group_size(uint32_t n_peers, double failure_rate, uint32_t max_group, uint32_t *m_out,
                                 double *expected_out) {
    if (!m_out || n_peers < 2 || n_peers > DEDLOC_MAX_GROUP_PEERS || !(failure_rate >= 0.0) ||
        !(failure_rate < 1.0) || max_group == 1)
        return DEDLOC_ERR_INVALID_ARG;
    const uint32_t hi = max_group ? std::min(max_group, n_peers) : n_peers;
    uint32_t best_m = 0;
    double best = INFINITY;
    for (uint32_t m = 2; m <= hi; m++) {
        uint32_t d = 1;
        uint64_t reach = m;
        while (reach < n_peers) {
            reach *= m;
            d++;
        }
        const double e = (double)d / pow(1.0 - failure_rate, (double)m);
        if (e < best) {
            best = e;
            best_m = m;
        }
    }
    *m_out = best_m;
    if (expected_out) *expected_out = best;
    return DEDLOC_OK;
}
