/*
 * birkhoffn_oracle.c -- fp64 CPU oracle for batched n x n Birkhoff projection,
 * n = 2 .. 16 (the mHC layer uses n = 4 or 8, Sec. 3.1).
 *
 * TEST INFRASTRUCTURE ONLY. The tests, the smoke check and the benchmark's
 * CPU-baseline leg load this library; the product path never does, and the two
 * share no code. It is independent of birkhoff4_oracle.c as well (a second,
 * size-generic implementation, so that the 4 x 4 case pins one against the other).
 *
 * Paper notation: R = H is the logit matrix, M = -R the cost, eta = 1 and
 * a = b = 1 (Sec. 2.3). One matrix at a time, row-major [n][n], double precision.
 *
 *   forward   P = T(beta*) with beta* minimising the reduced dual f (eq. min_fx) over
 *             x = beta_{-m} (m = n), by damped Newton (Sec. 3.1) with the gradient
 *             and Hessian of eq. grad_hess (a = 1, eta = 1):
 *               grad f = c_{-m} - 1,   hess f = diag(c_{-m}) - T_{-m}^T T_{-m},
 *             c = T^T 1 the column sums, T the row softmax of H + 1 beta^T.
 *   dual      alpha* = alpha*(beta*) (eq. alpha_opt) and beta* with beta_n = 0.
 *   backward  dH = -D with D from eq. derivative (a = b = 1, eta = 1).
 *   sinkhorn  iterations of eq. sinkhorn_knopp run to a marginal tolerance (a
 *             second algorithm for the same projection, used by the pins).
 *
 * Readings (the same choices as the 4 x 4 oracle, written for general n):
 *  - x^(0) = 0;
 *  - the Hessian diagonal c_j - sum_i T_ij^2 is written as sum_{k != j} W_jk with
 *    W_jk = sum_i T_ij T_ik (unit row sums), so the Hessian is the Laplacian of
 *    the column graph with weights W grounded at column n; the Newton system gets
 *    a Levenberg-Marquardt shift 1e-6 max_j |g_j| and is solved by eliminating
 *    nodes in natural order with pivots that are sums of positive weights;
 *  - Armijo backtracking (c1 = 1e-4, halving, 40 at most) from a step capped at
 *    |d|_inf <= 50; when f cannot resolve the decrease a step that lowers
 *    max_j |c_j - 1| is taken; otherwise one block-coordinate sweep (eq. bca);
 *  - stop: max over all n columns of |c_j - 1| <= tol, tested before each step;
 *  - the column sums near a permutation are formed without cancellation: for
 *    the dominant entry of a row, 1 - T_{i,dom} = sum_{k != dom} T_ik;
 *  - backward: mu_c - T_{-m}^T mu_r = sum_{k != j} F_jk with antisymmetric edge
 *    flows F_jk = sum_i T_ij T_ik (G_ij - G_ik), carried through the same
 *    elimination, and D_ij = -T_ij sum_{k != j} T_ik (psi_ij - psi_ik),
 *    psi = G - 1 w^T (identical given unit row sums, Sec. 4.1).
 */
#include <math.h>
#include <stdint.h>

#define NMAX 16
#define CAP 50.0
#define ARMIJO 1e-4
#define LM 1e-6

/* T = row softmax of H + 1 beta^T; lse_i = log sum_j exp(H_ij + beta_j) (so
 * alpha*_i = -lse_i, eq. alpha_opt); dom_i the first column attaining the row max */
static void evaluate(int n, const double *H, const double *beta, double *T, double *lse,
                     int *dom)
{
    for (int i = 0; i < n; ++i) {
        double U[NMAX], mu = -INFINITY, s = 0.0;
        dom[i] = 0;
        for (int j = 0; j < n; ++j) {
            U[j] = H[n * i + j] + beta[j];
            if (U[j] > mu) { mu = U[j]; dom[i] = j; }
        }
        for (int j = 0; j < n; ++j) s += exp(U[j] - mu);
        for (int j = 0; j < n; ++j) T[n * i + j] = exp(U[j] - mu) / s;
        lse[i] = mu + log(s);
    }
}

/* g_j = c_j - 1 for all n columns, without cancellation (see the readings) */
static void gradient(int n, const double *T, const int *dom, double *g)
{
    for (int j = 0; j < n; ++j) {
        double s = -1.0;
        for (int i = 0; i < n; ++i) {
            if (dom[i] == j) {
                s += 1.0;
                for (int k = 0; k < n; ++k)
                    if (k != j) s -= T[n * i + k];
            } else {
                s += T[n * i + j];
            }
        }
        g[j] = s;
    }
}

static double max_abs(int n, const double *g)
{
    double r = 0.0;
    for (int j = 0; j < n; ++j) {
        double e = fabs(g[j]);
        if (!(e <= r)) r = e; /* NaN propagates */
    }
    return r;
}

/* W_jk = sum_i T_ij T_ik */
static void weights(int n, const double *T, double W[NMAX][NMAX])
{
    for (int j = 0; j < n; ++j)
        for (int k = 0; k < n; ++k) {
            double s = 0.0;
            for (int i = 0; i < n; ++i) s += T[n * i + j] * T[n * i + k];
            W[j][k] = s;
        }
}

/* Solve (L + shift I) x = r, L the Laplacian of nodes 0 .. n-2 with weights W
 * and node n-1 the ground. Eliminating node p adds W_jp W_pk / piv_p to the edge
 * (j, k) and moves W_jp leak_p / piv_p of node p's leak to ground onto node j;
 * piv_p = sum of node p's remaining weights plus its leak. A node with no
 * conductance left gets x = 0. */
static void laplacian_solve(int n, double W[NMAX][NMAX], double shift, const double *r_in,
                            double *x)
{
    const int m = n - 1;
    double leak[NMAX], r[NMAX], piv[NMAX];
    for (int j = 0; j < m; ++j) {
        leak[j] = W[j][m] + shift;
        r[j] = r_in[j];
    }
    for (int p = 0; p < m; ++p) {
        piv[p] = leak[p];
        for (int k = p + 1; k < m; ++k) piv[p] += W[p][k];
        if (!(piv[p] > 0.0)) continue;
        for (int j = p + 1; j < m; ++j) {
            const double f = W[j][p] / piv[p];
            for (int k = j + 1; k < m; ++k) {
                W[j][k] += f * W[p][k];
                W[k][j] = W[j][k];
            }
            leak[j] += f * leak[p];
            r[j] += f * r[p];
        }
    }
    for (int p = m - 1; p >= 0; --p) {
        if (!(piv[p] > 0.0)) { x[p] = 0.0; continue; }
        double s = r[p];
        for (int k = p + 1; k < m; ++k) s += W[p][k] * x[k];
        x[p] = s / piv[p];
    }
}

static int all_finite(const double *x, int k)
{
    for (int q = 0; q < k; ++q)
        if (!isfinite(x[q])) return 0;
    return 1;
}

/* One projection; returns the number of updates, -1 if max_iter updates did not
 * reach tol, -2 for a non-finite input. dual = (alpha_1..alpha_n, beta_1..beta_n). */
static int project_one(int n, const double *H, double *P, double *dual, double tol, int max_iter)
{
    const int m = n - 1;
    if (!all_finite(H, n * n)) {
        for (int q = 0; q < n * n; ++q) P[q] = NAN;
        for (int q = 0; q < 2 * n; ++q) dual[q] = NAN;
        return -2;
    }
    double beta[NMAX] = {0.0}, T[NMAX * NMAX], lse[NMAX], g[NMAX];
    int dom[NMAX], it = 0, converged = 0;
    evaluate(n, H, beta, T, lse, dom);
    gradient(n, T, dom, g);
    for (;;) {
        const double res = max_abs(n, g);
        if (res <= tol) { converged = 1; break; }
        if (it >= max_iter) break;

        double W[NMAX][NMAX], rhs[NMAX], d[NMAX];
        weights(n, T, W);
        for (int j = 0; j < m; ++j) rhs[j] = -g[j];
        laplacian_solve(n, W, LM * res, rhs, d);
        double dmax = 0.0;
        for (int j = 0; j < m; ++j) dmax = fmax(dmax, fabs(d[j]));
        if (dmax > CAP)
            for (int j = 0; j < m; ++j) d[j] *= CAP / dmax;
        double slope = 0.0, gn2 = 0.0, dn2 = 0.0;
        for (int j = 0; j < m; ++j) {
            slope += g[j] * d[j];
            gn2 += g[j] * g[j];
            dn2 += d[j] * d[j];
        }
        double fscale = 1.0;
        for (int i = 0; i < n; ++i) fscale += fabs(lse[i]);
        for (int j = 0; j < m; ++j) fscale += fabs(beta[j]);

        double bn[NMAX];
        int accepted = 0;
        if (slope < -1e-12 * sqrt(gn2 * dn2)) {
            double t = 1.0, Tn[NMAX * NMAX], ln[NMAX], gn[NMAX];
            int dn[NMAX];
            for (int bt = 0; bt < 40 && !accepted; ++bt, t *= 0.5) {
                for (int j = 0; j < m; ++j) bn[j] = beta[j] + t * d[j];
                bn[m] = 0.0;
                evaluate(n, H, bn, Tn, ln, dn);
                gradient(n, Tn, dn, gn);
                /* f(beta) = n + sum_i lse_i - sum_j beta_j (eq. min_fx, a = b = 1) */
                double df = 0.0;
                for (int i = 0; i < n; ++i) df += ln[i] - lse[i];
                for (int j = 0; j < m; ++j) df -= t * d[j];
                if (df <= ARMIJO * t * slope) accepted = 1;
                else if (fabs(df) <= 1e-13 * fscale && max_abs(n, gn) < res) accepted = 1;
            }
        }
        if (accepted) {
            for (int j = 0; j < n; ++j) beta[j] = bn[j];
        } else {
            /* beta <- beta*(alpha*(beta)) (eq. bca, eq. beta_opt), gauge beta_n = 0 */
            for (int j = 0; j < n; ++j) {
                double mu = -INFINITY, s = 0.0;
                for (int i = 0; i < n; ++i) mu = fmax(mu, H[n * i + j] - lse[i]);
                for (int i = 0; i < n; ++i) s += exp(H[n * i + j] - lse[i] - mu);
                bn[j] = -(mu + log(s));
            }
            for (int j = 0; j < n; ++j) beta[j] = bn[j] - bn[m];
        }
        ++it;
        evaluate(n, H, beta, T, lse, dom);
        gradient(n, T, dom, g);
    }
    for (int q = 0; q < n * n; ++q) P[q] = T[q];
    for (int i = 0; i < n; ++i) dual[i] = -lse[i];
    for (int j = 0; j < n; ++j) dual[n + j] = beta[j];
    return converged ? it : -1;
}

/* Elimination of nodes 0 .. n-2 of the grounded column Laplacian (weights W,
 * ground n-1) with the right-hand side carried as antisymmetric edge flows:
 * eliminating p joins j, k by W_jp W_pk / piv and moves p's flows onto that edge,
 * F'_jk = F_jk + (W_pk F_jp + W_jp F_pk) / piv, piv = sum_{k > p} W_pk. Then
 * w_p = sum_{k > p} (W_pk w_k + F_pk) / piv, w_{n-1} = 0. */
static void laplacian_solve_flows(int n, double W[NMAX][NMAX], double F[NMAX][NMAX], double *w)
{
    const int m = n - 1;
    double piv[NMAX];
    for (int p = 0; p < m; ++p) {
        piv[p] = 0.0;
        for (int k = p + 1; k < n; ++k) piv[p] += W[p][k];
        if (!(piv[p] > 0.0)) continue;
        for (int j = p + 1; j < n; ++j)
            for (int k = j + 1; k < n; ++k) {
                const double Wn = W[j][k] + W[j][p] * W[p][k] / piv[p];
                const double Fn = F[j][k] + (W[p][k] * F[j][p] + W[j][p] * F[p][k]) / piv[p];
                W[j][k] = W[k][j] = Wn;
                F[j][k] = Fn;
                F[k][j] = -Fn;
            }
    }
    w[m] = 0.0;
    for (int p = m - 1; p >= 0; --p) {
        if (!(piv[p] > 0.0)) { w[p] = 0.0; continue; }
        double s = 0.0;
        for (int k = p + 1; k < n; ++k) s += W[p][k] * w[k] + F[p][k];
        w[p] = s / piv[p];
    }
}

static void backward_one(int n, const double *T, const double *G, double *dH)
{
    double W[NMAX][NMAX], F[NMAX][NMAX], w[NMAX];
    weights(n, T, W);
    for (int j = 0; j < n; ++j)
        for (int k = 0; k < n; ++k) {
            double s = 0.0;
            for (int i = 0; i < n; ++i)
                s += T[n * i + j] * T[n * i + k] * (G[n * i + j] - G[n * i + k]);
            F[j][k] = s;
        }
    laplacian_solve_flows(n, W, F, w);
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j) {
            const double psi_ij = G[n * i + j] - w[j];
            double s = 0.0;
            for (int k = 0; k < n; ++k)
                if (k != j) s += T[n * i + k] * (psi_ij - (G[n * i + k] - w[k]));
            dH[n * i + j] = T[n * i + j] * s; /* -D, R = -M */
        }
}

/* Sinkhorn-Knopp (eq. sinkhorn_knopp) on A = exp(H - max H), v^(0) = 1, run until
 * the row sums of diag(u) A diag(v) are within tol of one (its column sums are
 * exact after each v update) or max_steps; returns the steps taken. */
static int sinkhorn_one(int n, const double *H, double *P, double tol, int max_steps)
{
    double A[NMAX * NMAX], u[NMAX], v[NMAX], mx = -INFINITY;
    for (int q = 0; q < n * n; ++q) mx = fmax(mx, H[q]);
    for (int q = 0; q < n * n; ++q) A[q] = exp(H[q] - mx);
    for (int j = 0; j < n; ++j) v[j] = 1.0;
    int steps = 0;
    for (; steps < max_steps; ++steps) {
        for (int i = 0; i < n; ++i) {
            double s = 0.0;
            for (int j = 0; j < n; ++j) s += A[n * i + j] * v[j];
            u[i] = 1.0 / s;
        }
        for (int j = 0; j < n; ++j) {
            double s = 0.0;
            for (int i = 0; i < n; ++i) s += A[n * i + j] * u[i];
            v[j] = 1.0 / s;
        }
        double err = 0.0; /* row sums (columns are exact after the v update) */
        for (int i = 0; i < n; ++i) {
            double s = 0.0;
            for (int j = 0; j < n; ++j) s += u[i] * A[n * i + j] * v[j];
            err = fmax(err, fabs(s - 1.0));
        }
        if (err <= tol) { ++steps; break; }
    }
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j) P[n * i + j] = u[i] * A[n * i + j] * v[j];
    return steps;
}

/* ---------------------------------------------------------------------------
 * Batched entry points (ranges [lo, hi) of matrices)
 * ------------------------------------------------------------------------- */
int oraclen_fwd(int n, const double *H, double *P, double *dual, int32_t *iters, int64_t lo,
                int64_t hi, double tol, int max_iter)
{
    if (n < 2 || n > NMAX) return -1;
    for (int64_t b = lo; b < hi; ++b)
        iters[b] = project_one(n, H + (int64_t)n * n * b, P + (int64_t)n * n * b,
                               dual + (int64_t)2 * n * b, tol, max_iter);
    return 0;
}

int oraclen_bwd(int n, const double *P, const double *G, double *dH, int64_t lo, int64_t hi)
{
    if (n < 2 || n > NMAX) return -1;
    for (int64_t b = lo; b < hi; ++b)
        backward_one(n, P + (int64_t)n * n * b, G + (int64_t)n * n * b, dH + (int64_t)n * n * b);
    return 0;
}

int oraclen_sinkhorn(int n, const double *H, double *P, int32_t *steps, int64_t lo, int64_t hi,
                     double tol, int max_steps)
{
    if (n < 2 || n > NMAX) return -1;
    for (int64_t b = lo; b < hi; ++b)
        steps[b] = sinkhorn_one(n, H + (int64_t)n * n * b, P + (int64_t)n * n * b, tol, max_steps);
    return 0;
}

/* ---------------------------------------------------------------------------
 * General entropic OT (eq. entropic): cost M, marginals a > 0, b > 0 with equal sums,
 * regulariser eta > 0. Dual eq. dual, partial maximiser eq. alpha_opt, reduced
 * problem eq. min_fx over x = beta_{-m}, gradient and Hessian eq. grad_hess:
 *   T_ij = a_i softmax_j((beta_j - M_ij) / eta),
 *   grad f = T_{-m}^T 1 - b_{-m},
 *   hess f = eta^{-1} (diag(c_{-m}) - T_{-m}^T diag(a)^{-1} T_{-m}),
 * whose diagonal c_j - sum_i T_ij^2 / a_i = sum_{k != j} W_jk with
 * W_jk = sum_i T_ij T_ik / a_i (rows of T sum to a_i): the grounded Laplacian of the
 * column graph again. The same damped Newton as for the projection, with
 * f(beta) = eta sum_i a_i - alpha*(beta)^T a - beta^T b and the stop test
 * max_j |c_j - b_j| <= tol. Backward: eq. derivative with
 *   mu_c - T_{-m}^T (mu_r / a) = sum_{k != j} F_jk,  F_jk = sum_i T_ij T_ik (G_ij - G_ik) / a_i,
 *   D_ij = -eta^{-1} T_ij (psi_ij - sum_k T_ik psi_ik / a_i),  psi = G - 1 w^T,
 * returned as dL/dM = D.
 * ------------------------------------------------------------------------- */

/* T_ij = a_i exp(U_ij - mu_i) / s_i with U_ij = (beta_j - M_ij) / eta; lse_i = mu_i + log s_i */
static void ot_evaluate(int n, const double *M, const double *a, double eta, const double *beta,
                        double *T, double *lse)
{
    for (int i = 0; i < n; ++i) {
        double U[NMAX], mu = -INFINITY, s = 0.0;
        for (int j = 0; j < n; ++j) {
            U[j] = (beta[j] - M[n * i + j]) / eta;
            if (U[j] > mu) mu = U[j];
        }
        for (int j = 0; j < n; ++j) s += exp(U[j] - mu);
        for (int j = 0; j < n; ++j) T[n * i + j] = a[i] * exp(U[j] - mu) / s;
        lse[i] = mu + log(s);
    }
}

/* g_j = c_j - b_j; near a permutation-like T the column sums are formed from the
 * small entries: for the dominant entry of row i, T_{i,dom} = a_i - sum_{k != dom} T_ik */
static void ot_gradient(int n, const double *T, const double *a, const double *b, double *g)
{
    int dom[NMAX];
    for (int i = 0; i < n; ++i) {
        dom[i] = 0;
        for (int j = 1; j < n; ++j)
            if (T[n * i + j] > T[n * i + dom[i]]) dom[i] = j;
    }
    for (int j = 0; j < n; ++j) {
        double s = -b[j];
        for (int i = 0; i < n; ++i) {
            if (dom[i] == j) {
                s += a[i];
                for (int k = 0; k < n; ++k)
                    if (k != j) s -= T[n * i + k];
            } else {
                s += T[n * i + j];
            }
        }
        g[j] = s;
    }
}

static int ot_one(int n, const double *M, const double *a, const double *b, double eta, double *T,
                  double *dual, double tol, int max_iter)
{
    const int m = n - 1;
    if (!all_finite(M, n * n) || !all_finite(a, n) || !all_finite(b, n)) {
        for (int q = 0; q < n * n; ++q) T[q] = NAN;
        for (int q = 0; q < 2 * n; ++q) dual[q] = NAN;
        return -2;
    }
    double beta[NMAX] = {0.0}, lse[NMAX], g[NMAX];
    int it = 0, converged = 0;
    ot_evaluate(n, M, a, eta, beta, T, lse);
    ot_gradient(n, T, a, b, g);
    for (;;) {
        const double res = max_abs(n, g);
        if (res <= tol) { converged = 1; break; }
        if (it >= max_iter) break;
        /* Newton direction d = -[hess f + lambda I]^{-1} grad f; hess f = L(W) / eta */
        double W[NMAX][NMAX], rhs[NMAX], d[NMAX];
        for (int j = 0; j < n; ++j)
            for (int k = 0; k < n; ++k) {
                double s = 0.0;
                for (int i = 0; i < n; ++i) s += T[n * i + j] * T[n * i + k] / a[i];
                W[j][k] = s / eta;
            }
        for (int j = 0; j < m; ++j) rhs[j] = -g[j];
        laplacian_solve(n, W, LM * res, rhs, d);
        double dmax = 0.0;
        for (int j = 0; j < m; ++j) dmax = fmax(dmax, fabs(d[j]));
        if (dmax > CAP * eta)
            for (int j = 0; j < m; ++j) d[j] *= CAP * eta / dmax;
        double slope = 0.0, gn2 = 0.0, dn2 = 0.0;
        for (int j = 0; j < m; ++j) {
            slope += g[j] * d[j];
            gn2 += g[j] * g[j];
            dn2 += d[j] * d[j];
        }
        double fscale = 1.0;
        for (int i = 0; i < n; ++i) fscale += fabs(eta * a[i] * lse[i]);
        for (int j = 0; j < m; ++j) fscale += fabs(b[j] * beta[j]);
        double bn[NMAX], Tn[NMAX * NMAX], ln[NMAX], gn[NMAX];
        int accepted = 0;
        if (slope < -1e-12 * sqrt(gn2 * dn2)) {
            double t = 1.0;
            for (int bt = 0; bt < 40 && !accepted; ++bt, t *= 0.5) {
                for (int j = 0; j < m; ++j) bn[j] = beta[j] + t * d[j];
                bn[m] = 0.0;
                ot_evaluate(n, M, a, eta, bn, Tn, ln);
                ot_gradient(n, Tn, a, b, gn);
                /* f = eta sum_i a_i (1 + lse_i - log a_i) - beta^T b: its change, row by row */
                double df = 0.0;
                for (int i = 0; i < n; ++i) df += eta * a[i] * (ln[i] - lse[i]);
                for (int j = 0; j < m; ++j) df -= b[j] * t * d[j];
                if (df <= ARMIJO * t * slope) accepted = 1;
                else if (fabs(df) <= 1e-13 * fscale && max_abs(n, gn) < res) accepted = 1;
            }
        }
        if (accepted) {
            for (int j = 0; j < n; ++j) beta[j] = bn[j];
        } else {
            /* beta <- beta*(alpha*(beta)) (eq. bca, eq. beta_opt), gauge beta_n = 0 */
            for (int j = 0; j < n; ++j) {
                double mu = -INFINITY, s = 0.0, al[NMAX];
                for (int i = 0; i < n; ++i) {
                    al[i] = eta * (log(a[i]) - lse[i]); /* alpha*_i(beta) */
                    mu = fmax(mu, (al[i] - M[n * i + j]) / eta);
                }
                for (int i = 0; i < n; ++i) s += exp((al[i] - M[n * i + j]) / eta - mu);
                bn[j] = eta * log(b[j]) - eta * (mu + log(s));
            }
            for (int j = 0; j < n; ++j) beta[j] = bn[j] - bn[m];
        }
        ++it;
        ot_evaluate(n, M, a, eta, beta, T, lse);
        ot_gradient(n, T, a, b, g);
    }
    for (int i = 0; i < n; ++i) dual[i] = eta * (log(a[i]) - lse[i]);
    for (int j = 0; j < n; ++j) dual[n + j] = beta[j];
    return converged ? it : -1;
}

static void ot_backward_one(int n, const double *T, const double *a, double eta, const double *G,
                            double *dM)
{
    double W[NMAX][NMAX], F[NMAX][NMAX], w[NMAX];
    for (int j = 0; j < n; ++j)
        for (int k = 0; k < n; ++k) {
            double sw = 0.0, sf = 0.0;
            for (int i = 0; i < n; ++i) {
                const double q = T[n * i + j] * T[n * i + k] / a[i];
                sw += q;
                sf += q * (G[n * i + j] - G[n * i + k]);
            }
            W[j][k] = sw;
            F[j][k] = sf;
        }
    laplacian_solve_flows(n, W, F, w); /* Delta w = mu_c - T^T (mu_r / a), Delta = L(W) */
    for (int i = 0; i < n; ++i) {
        double s = 0.0;
        for (int k = 0; k < n; ++k) s += T[n * i + k] * (G[n * i + k] - w[k]);
        s /= a[i];
        for (int j = 0; j < n; ++j)
            dM[n * i + j] = -T[n * i + j] * ((G[n * i + j] - w[j]) - s) / eta;
    }
}

/* Sinkhorn with marginals: u = a / (K v), v = b / (K^T u), K = exp(-(M - min M) / eta) */
static int ot_sinkhorn_one(int n, const double *M, const double *a, const double *b, double eta,
                           double *T, double tol, int max_steps)
{
    double K[NMAX * NMAX], u[NMAX], v[NMAX], mn = INFINITY;
    for (int q = 0; q < n * n; ++q) mn = fmin(mn, M[q]);
    for (int q = 0; q < n * n; ++q) K[q] = exp(-(M[q] - mn) / eta);
    for (int j = 0; j < n; ++j) v[j] = 1.0;
    int steps = 0;
    for (; steps < max_steps; ++steps) {
        for (int i = 0; i < n; ++i) {
            double s = 0.0;
            for (int j = 0; j < n; ++j) s += K[n * i + j] * v[j];
            u[i] = a[i] / s;
        }
        for (int j = 0; j < n; ++j) {
            double s = 0.0;
            for (int i = 0; i < n; ++i) s += K[n * i + j] * u[i];
            v[j] = b[j] / s;
        }
        double err = 0.0;
        for (int i = 0; i < n; ++i) {
            double s = 0.0;
            for (int j = 0; j < n; ++j) s += u[i] * K[n * i + j] * v[j];
            err = fmax(err, fabs(s - a[i]));
        }
        if (err <= tol) { ++steps; break; }
    }
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j) T[n * i + j] = u[i] * K[n * i + j] * v[j];
    return steps;
}

int oraclen_ot_fwd(int n, const double *M, const double *a, const double *b, double eta, double *T,
                   double *dual, int32_t *iters, int64_t lo, int64_t hi, double tol, int max_iter)
{
    if (n < 2 || n > NMAX || !(eta > 0.0)) return -1;
    for (int64_t q = lo; q < hi; ++q)
        iters[q] = ot_one(n, M + (int64_t)n * n * q, a + (int64_t)n * q, b + (int64_t)n * q, eta,
                          T + (int64_t)n * n * q, dual + (int64_t)2 * n * q, tol, max_iter);
    return 0;
}

int oraclen_ot_bwd(int n, const double *T, const double *a, double eta, const double *G, double *dM,
                   int64_t lo, int64_t hi)
{
    if (n < 2 || n > NMAX || !(eta > 0.0)) return -1;
    for (int64_t q = lo; q < hi; ++q)
        ot_backward_one(n, T + (int64_t)n * n * q, a + (int64_t)n * q, eta, G + (int64_t)n * n * q,
                        dM + (int64_t)n * n * q);
    return 0;
}

int oraclen_ot_sinkhorn(int n, const double *M, const double *a, const double *b, double eta,
                        double *T, int32_t *steps, int64_t lo, int64_t hi, double tol, int max_steps)
{
    if (n < 2 || n > NMAX || !(eta > 0.0)) return -1;
    for (int64_t q = lo; q < hi; ++q)
        steps[q] = ot_sinkhorn_one(n, M + (int64_t)n * n * q, a + (int64_t)n * q, b + (int64_t)n * q,
                                   eta, T + (int64_t)n * n * q, tol, max_steps);
    return 0;
}
