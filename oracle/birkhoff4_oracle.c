/*
 * birkhoff4_oracle.c -- fp64 CPU oracle for the batched 4x4 Birkhoff projection.
 *
 * TEST INFRASTRUCTURE ONLY. The tests, the smoke check and the benchmark's
 * CPU-baseline leg load this library; the product path (the HIP library and its
 * Python binding) never does, and the two share no code.
 *
 * Paper notation: R = H is the logit matrix, M = -R the cost, eta = 1 and
 * a = b = 1 (Sec. 2.3: the Birkhoff projection of exp(R) is entropic OT with
 * these parameters). Every routine works on one matrix at a time, row-major
 * [4][4], in double precision, with no blocking or vectorisation.
 *
 *   forward   P = argmin over the Birkhoff polytope of KL(P || exp H)
 *             (eq. birkhoff_projection), reached as P = T(beta*) where beta*
 *             minimises the reduced dual f (eq. min_fx) by damped Newton
 *             (Sec. 3.1) with the 4x4 gradient and Hessian (Sec. 3.2).
 *   dual      alpha* = alpha*(beta*) (eq. alpha_opt) and beta* with beta_4 = 0.
 *   backward  dH = -D with D from eq. derivative, specialised to 4x4 (Sec. 4.2).
 *   baseline  n steps of Sinkhorn-Knopp (eq. sinkhorn_knopp) and the exact
 *             reverse-mode gradient of that n-step map.
 *
 * Readings where the text leaves a choice:
 *  - initial point x^(0) = 0 (the paper gives none);
 *  - Newton direction with a Levenberg-Marquardt shift 1e-6 max_j |g_j| on the
 *    Hessian diagonal (zero at the solution; see newton_direction);
 *  - step size: Armijo backtracking on f (c1 = 1e-4, halving) from a Newton
 *    step capped at |d|_inf <= 50. When f can no longer resolve the decrease
 *    (|delta f| at rounding level) a step that lowers max_j |c_j - 1| is taken;
 *    if the capped Newton direction is not a descent direction (angle test) or
 *    backtracking reaches no acceptable step within 40 halvings, one
 *    block-coordinate sweep
 *    beta <- beta*(alpha*(beta)) (eq. bca) is taken instead;
 *  - stop: max over all four columns of |c_j - 1| <= tol, tested before each
 *    step (rows sum to one by construction);
 *  - the Hessian diagonal c_j - sum_i T_ij^2 is written as
 *    sum_i T_ij sum_{k != j} T_ik (equal because every row of T sums to one),
 *    so the Hessian is the Laplacian of the column graph with weights
 *    sum_i T_ij T_ik, grounded at column 4, and the 3x3 system is solved by
 *    Gaussian elimination whose pivots are sums of these positive weights;
 *  - backward: the right-hand side mu_c - T_{-m}^T mu_r and the entries of D are
 *    evaluated in rearranged forms that are algebraically identical given unit
 *    row sums (written next to each formula), so that nothing cancels when P
 *    is close to a permutation.
 */
#include <math.h>
#include <stdint.h>

#define ORACLE_CAP 50.0
#define ORACLE_ARMIJO 1e-4
#define ORACLE_LM 1e-6

/* ---------------------------------------------------------------------------
 * Forward pieces
 * ------------------------------------------------------------------------- */

/* Row-softmax evaluation at beta (Sec. 3.2): U_ij = beta_j + H_ij,
 * T_ij = exp(U_ij - mu_i) / sum_k exp(U_ik - mu_i) with mu_i = max_j U_ij
 * (eq. tij_stable), alpha_i = -log sum_j exp(U_ij) (eq. alpha_opt, a_i = 1).
 * lse[i] receives log sum_j exp(U_ij) = mu_i + log s_i, dom[i] the first column
 * attaining mu_i. */
static void evaluate(const double H[16], const double beta[4], double T[16],
                     double alpha[4], double lse[4], int dom[4])
{
    for (int i = 0; i < 4; ++i) {
        double U[4], mu = -INFINITY, s = 0.0;
        dom[i] = 0;
        for (int j = 0; j < 4; ++j) {
            U[j] = beta[j] + H[4 * i + j];
            if (U[j] > mu) { mu = U[j]; dom[i] = j; }
        }
        for (int j = 0; j < 4; ++j) s += exp(U[j] - mu);
        for (int j = 0; j < 4; ++j) T[4 * i + j] = exp(U[j] - mu) / s;
        lse[i] = mu + log(s);
        alpha[i] = -lse[i];
    }
}

/* Gradient of f extended to all four columns, g_j = c_j - 1 with
 * c_j = sum_i T_ij (eq. c_g). Written without cancellation: for the dominant
 * entry of row i, 1 - T_{i,dom(i)} = sum_{k != dom(i)} T_ik (unit row sums), so
 *   g_j = (n_j - 1) + sum_{i: dom(i) != j} T_ij - sum_{i: dom(i) = j} sum_{k != j} T_ik
 * with n_j the number of rows whose dominant column is j. Every term is then
 * small when T is close to a permutation and is computed to full relative
 * accuracy, and sum_j g_j = 0 holds to that accuracy. */
static void marginal_gradient(const double T[16], const int dom[4], double g[4])
{
    for (int j = 0; j < 4; ++j) {
        double s = -1.0;
        for (int i = 0; i < 4; ++i)
            if (dom[i] == j) s += 1.0;
        for (int i = 0; i < 4; ++i) {
            if (dom[i] != j) s += T[4 * i + j];
            else
                for (int k = 0; k < 4; ++k)
                    if (k != j) s -= T[4 * i + k];
        }
        g[j] = s;
    }
}

static double max_abs4(const double g[4])
{
    double r = 0.0;
    for (int j = 0; j < 4; ++j) {
        double e = fabs(g[j]);
        if (!(e <= r)) r = e; /* NaN propagates */
    }
    return r;
}

/* Column-graph weights w_jk = sum_i T_ij T_ik = l_j^T l_k (the p_jk of Sec. 3.2,
 * extended to the fourth column). The Hessian of f is
 *   h_jk = -w_jk (j != k),   h_jj = c_j - p_jj = sum_{k != j} w_jk   (j,k <= 3). */
static void column_weights(const double T[16], double w[4][4])
{
    for (int j = 0; j < 4; ++j)
        for (int k = 0; k < 4; ++k) {
            double s = 0.0;
            for (int i = 0; i < 4; ++i) s += T[4 * i + j] * T[4 * i + k];
            w[j][k] = s;
        }
}

/* Solve (L + shift I) x = r for the Laplacian L of nodes {0,1,2} with edge
 * weights w[j][k] (j,k in 0..3, node 3 is the ground); the shift acts as an
 * extra conductance from every node to the ground. Gaussian elimination in natural
 * order; each pivot is the sum of the remaining weights of its node, which is
 * what subtraction would give in exact arithmetic. A node whose pivot is zero
 * has no conductance left and gets x = 0 (its equation carries no information). */
static void laplacian_solve(const double w[4][4], double shift, const double r_in[3],
                            double x[3])
{
    double a[3][3], gnd[3], r[3], piv[3];
    for (int j = 0; j < 3; ++j) {
        for (int k = 0; k < 3; ++k) a[j][k] = (j == k) ? 0.0 : w[j][k];
        gnd[j] = w[j][3] + shift;
        r[j] = r_in[j];
    }
    for (int p = 0; p < 3; ++p) {
        piv[p] = gnd[p];
        for (int k = p + 1; k < 3; ++k) piv[p] += a[p][k];
        if (!(piv[p] > 0.0)) continue;
        for (int j = p + 1; j < 3; ++j) {
            double f = a[j][p] / piv[p];
            for (int k = p + 1; k < 3; ++k)
                if (k != j) a[j][k] += f * a[p][k];
            gnd[j] += f * gnd[p];
            r[j] += f * r[p];
        }
    }
    for (int p = 2; p >= 0; --p) {
        if (!(piv[p] > 0.0)) { x[p] = 0.0; continue; }
        double s = r[p];
        for (int k = p + 1; k < 3; ++k) s += a[p][k] * x[k];
        x[p] = s / piv[p];
    }
}

/* Newton direction d = -[nabla^2 f + lambda I]^{-1} nabla f at the evaluated T
 * (Sec. 3.1), with lambda = ORACLE_LM * max_j |g_j|. The shift vanishes at the
 * solution; away from it, it bounds the effect of rounding in the gradient on
 * directions in which the Hessian is numerically singular (tiny weights). */
static void newton_direction(const double T[16], const double g[4], double d[3])
{
    double w[4][4], rhs[3];
    column_weights(T, w);
    for (int j = 0; j < 3; ++j) rhs[j] = -g[j];
    laplacian_solve(w, ORACLE_LM * max_abs4(g), rhs, d);
}

static int all_finite(const double *x, int n)
{
    for (int k = 0; k < n; ++k)
        if (!isfinite(x[k])) return 0;
    return 1;
}

/* One projection. Returns the number of updates applied, -1 when max_iter
 * updates did not reach tol, -2 for a non-finite input. */
static int project_one(const double H[16], double P[16], double dual[8], double tol,
                       int max_iter)
{
    if (!all_finite(H, 16)) {
        for (int k = 0; k < 16; ++k) P[k] = NAN;
        for (int k = 0; k < 8; ++k) dual[k] = NAN;
        return -2;
    }
    double beta[4] = {0.0, 0.0, 0.0, 0.0}; /* x^(0) = 0, beta_4 = 0 (Sec. 3.1) */
    double T[16], alpha[4], lse[4], g[4];
    int dom[4];
    int it = 0, converged = 0;
    evaluate(H, beta, T, alpha, lse, dom);
    marginal_gradient(T, dom, g);
    for (;;) {
        double res = max_abs4(g);
        if (res <= tol) { converged = 1; break; }
        if (it >= max_iter) break;

        double d[3];
        newton_direction(T, g, d);
        double dmax = fmax(fabs(d[0]), fmax(fabs(d[1]), fabs(d[2])));
        if (dmax > ORACLE_CAP)
            for (int j = 0; j < 3; ++j) d[j] *= ORACLE_CAP / dmax;
        double slope = 0.0, gn2 = 0.0, dn2 = 0.0; /* g^T d, |g|^2, |d|^2 */
        for (int j = 0; j < 3; ++j) {
            slope += g[j] * d[j];
            gn2 += g[j] * g[j];
            dn2 += d[j] * d[j];
        }
        double fscale = 1.0;
        for (int i = 0; i < 4; ++i) fscale += fabs(lse[i]);
        for (int j = 0; j < 3; ++j) fscale += fabs(beta[j]);

        int accepted = 0;
        double bn[4];
        /* A usable Newton direction points downhill; when the Hessian is
         * numerically singular next to an O(1) gradient it need not. */
        if (slope < -1e-12 * sqrt(gn2 * dn2)) {
            double t = 1.0, Tn[16], an[4], ln[4], gn[4];
            int dn[4];
            for (int bt = 0; bt < 40 && !accepted; ++bt, t *= 0.5) {
                for (int j = 0; j < 3; ++j) bn[j] = beta[j] + t * d[j];
                bn[3] = 0.0;
                evaluate(H, bn, Tn, an, ln, dn);
                marginal_gradient(Tn, dn, gn);
                /* f(beta) = 4 + sum_i lse_i - sum_j beta_j (eq. min_fx); the
                 * change is accumulated row by row so it is not lost against |f| */
                double df = 0.0;
                for (int i = 0; i < 4; ++i) df += ln[i] - lse[i];
                for (int j = 0; j < 3; ++j) df -= t * d[j];
                if (df <= ORACLE_ARMIJO * t * slope) accepted = 1;
                else if (fabs(df) <= 1e-13 * fscale && max_abs4(gn) < res) accepted = 1;
            }
        }
        if (accepted) {
            for (int j = 0; j < 4; ++j) beta[j] = bn[j];
        } else {
            /* block-coordinate sweep: beta_j = beta*_j(alpha) of eq. beta_opt at
             * alpha = alpha*(beta), i.e. -log sum_i exp(alpha_i + H_ij), taken in
             * the log domain; then the gauge beta_4 = 0 is restored */
            for (int j = 0; j < 4; ++j) {
                double m = -INFINITY, s = 0.0;
                for (int i = 0; i < 4; ++i) m = fmax(m, alpha[i] + H[4 * i + j]);
                for (int i = 0; i < 4; ++i) s += exp(alpha[i] + H[4 * i + j] - m);
                bn[j] = -(m + log(s));
            }
            for (int j = 0; j < 4; ++j) beta[j] = bn[j] - bn[3];
        }
        ++it;
        evaluate(H, beta, T, alpha, lse, dom);
        marginal_gradient(T, dom, g);
    }
    for (int k = 0; k < 16; ++k) P[k] = T[k];
    for (int i = 0; i < 4; ++i) dual[i] = alpha[i];
    for (int j = 0; j < 4; ++j) dual[4 + j] = beta[j];
    return converged ? it : -1;
}

/* Solve Delta w = r with Delta the Laplacian of columns {0,1,2} grounded at
 * column 3 (edge weights W), when the right-hand side is a sum of antisymmetric
 * edge flows, r_j = sum_{k != j} F_jk with F_kj = -F_jk. Gaussian elimination of
 * nodes 0 and 1 in turn; eliminating node p joins its neighbours j, k by an
 * edge of weight W_jp W_pk / piv and moves its flows onto the same edges,
 *   F'_jk = F_jk + (W_pk F_jp + W_jp F_pk) / piv,   piv = sum_k W_pk,
 * which is the same elimination written so that every right-hand side stays a
 * sum of edge flows (no rounding can leak into a weakly connected node). A node
 * with zero pivot is disconnected and gets w = 0. w[3] = 0. */
static void laplacian_solve_flows(double W[4][4], double F[4][4], double w[4])
{
    double piv[3];
    for (int p = 0; p < 3; ++p) {
        piv[p] = 0.0;
        for (int k = p + 1; k < 4; ++k) piv[p] += W[p][k];
        if (!(piv[p] > 0.0) || p == 2) continue;
        for (int j = p + 1; j < 4; ++j)
            for (int k = p + 1; k < 4; ++k) {
                if (k == j) continue;
                if (k < j) continue; /* update each unordered pair once */
                double Wn = W[j][k] + W[j][p] * W[p][k] / piv[p];
                double Fn = F[j][k] + (W[p][k] * F[j][p] + W[j][p] * F[p][k]) / piv[p];
                W[j][k] = W[k][j] = Wn;
                F[j][k] = Fn;
                F[k][j] = -Fn;
            }
    }
    w[3] = 0.0;
    for (int p = 2; p >= 0; --p) {
        if (!(piv[p] > 0.0)) { w[p] = 0.0; continue; }
        double s = 0.0;
        for (int k = p + 1; k < 4; ++k) s += W[p][k] * w[k] + F[p][k];
        w[p] = s / piv[p];
    }
}

/* ---------------------------------------------------------------------------
 * Backward (Sec. 4.2, eq. derivative with eta = 1, a = b = 1)
 * ------------------------------------------------------------------------- */
static void implicit_backward_one(const double T[16], const double G[16], double dH[16])
{
    double W[4][4], F[4][4], w[4];
    /* Gamma = G o T*, mu_r = Gamma 1, mu_c = Gamma^T 1. The right-hand side
     *   mu_c,j - sum_i T_ij mu_r,i = sum_{k != j} F_jk,
     *   F_jk = sum_i T_ij T_ik (G_ij - G_ik)                (unit row sums),
     * and Delta = diag(b_{-m}) - T^T T is taken as the Hessian at T*, the
     * Laplacian with weights W_jk = sum_i T_ij T_ik. */
    column_weights(T, W);
    for (int j = 0; j < 4; ++j)
        for (int k = 0; k < 4; ++k) {
            double s = 0.0;
            for (int i = 0; i < 4; ++i)
                s += T[4 * i + j] * T[4 * i + k] * (G[4 * i + j] - G[4 * i + k]);
            F[j][k] = s;
        }
    laplacian_solve_flows(W, F, w); /* w_{-m} = Delta^{-1}(...), w_4 = 0 */
    /* v_i = mu_r,i - sum_j T_ij w_j and D_ij = (v_i + w_j - G_ij) T_ij,
     * i.e. D_ij = -T_ij sum_{k != j} T_ik (psi_ij - psi_ik), psi = G - 1 w^T */
    for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) {
            double psi_ij = G[4 * i + j] - w[j], s = 0.0;
            for (int k = 0; k < 4; ++k) {
                if (k == j) continue;
                s += T[4 * i + k] * (psi_ij - (G[4 * i + k] - w[k]));
            }
            double D = -T[4 * i + j] * s;
            dH[4 * i + j] = -D; /* R = -M flips the sign (Sec. 4.2) */
        }
}

/* ---------------------------------------------------------------------------
 * n-step Sinkhorn-Knopp (eq. sinkhorn_knopp) and its reverse-mode gradient.
 * A = exp(H) with each row shifted by its maximum: the first u-update absorbs
 * any row scaling of A, so every iterate's diag(u) A diag(v) is unchanged.
 * v^(0) = 1. Output diag(u^(n)) A diag(v^(n)).
 * ------------------------------------------------------------------------- */
#define SK_MAX_STEPS 256

static void sk_row_scaled_kernel(const double H[16], double A[16])
{
    for (int i = 0; i < 4; ++i) {
        double m = H[4 * i];
        for (int j = 1; j < 4; ++j) m = fmax(m, H[4 * i + j]);
        for (int j = 0; j < 4; ++j) A[4 * i + j] = exp(H[4 * i + j] - m);
    }
}

static void sk_forward_one(const double A[16], int n, double u[][4], double v[][4])
{
    for (int j = 0; j < 4; ++j) v[0][j] = 1.0;
    for (int k = 1; k <= n; ++k) {
        for (int i = 0; i < 4; ++i) {
            double s = 0.0;
            for (int j = 0; j < 4; ++j) s += A[4 * i + j] * v[k - 1][j];
            u[k][i] = 1.0 / s;
        }
        for (int j = 0; j < 4; ++j) {
            double s = 0.0;
            for (int i = 0; i < 4; ++i) s += A[4 * i + j] * u[k][i];
            v[k][j] = 1.0 / s;
        }
    }
}

/* ---------------------------------------------------------------------------
 * Exported entry points (batched loops; B matrices, row-major [B][4][4])
 * ------------------------------------------------------------------------- */
int oracle_fwd(const double *H, double *P, double *dual, int32_t *iters, int64_t B,
               double tol, int max_iter)
{
    int bad = 0;
    for (int64_t b = 0; b < B; ++b) {
        int it = project_one(H + 16 * b, P + 16 * b, dual + 8 * b, tol, max_iter);
        if (iters) iters[b] = it;
        if (it < 0) ++bad;
    }
    return bad;
}

void oracle_bwd(const double *P, const double *dP, double *dH, int64_t B)
{
    for (int64_t b = 0; b < B; ++b) implicit_backward_one(P + 16 * b, dP + 16 * b, dH + 16 * b);
}

int oracle_sk_fwd(const double *H, double *P, int64_t B, int n_steps)
{
    if (n_steps < 0 || n_steps > SK_MAX_STEPS) return -1;
    double u[SK_MAX_STEPS + 1][4], v[SK_MAX_STEPS + 1][4], A[16];
    for (int64_t b = 0; b < B; ++b) {
        sk_row_scaled_kernel(H + 16 * b, A);
        sk_forward_one(A, n_steps, u, v);
        for (int i = 0; i < 4; ++i)
            for (int j = 0; j < 4; ++j)
                P[16 * b + 4 * i + j] =
                    (n_steps == 0 ? 1.0 : u[n_steps][i]) * A[4 * i + j] * v[n_steps][j];
    }
    return 0;
}

/* Reverse mode through u^(k) = 1 / (A v^(k-1)), v^(k) = 1 / (A^T u^(k)),
 * P = diag(u^(n)) A diag(v^(n)), A_ij = exp(H_ij - max_k H_ik). Because P does
 * not depend on the row shift, dH_ij = Abar_ij A_ij exactly. */
int oracle_sk_bwd(const double *H, const double *dP, double *dH, int64_t B, int n_steps)
{
    if (n_steps < 1 || n_steps > SK_MAX_STEPS) return -1;
    double u[SK_MAX_STEPS + 1][4], v[SK_MAX_STEPS + 1][4], A[16];
    for (int64_t b = 0; b < B; ++b) {
        const double *G = dP + 16 * b;
        double Abar[16], ubar[4] = {0}, vbar[4] = {0};
        sk_row_scaled_kernel(H + 16 * b, A);
        sk_forward_one(A, n_steps, u, v);
        const int n = n_steps;
        for (int i = 0; i < 4; ++i)
            for (int j = 0; j < 4; ++j) {
                double g = G[4 * i + j];
                Abar[4 * i + j] = g * u[n][i] * v[n][j];
                ubar[i] += g * A[4 * i + j] * v[n][j];
                vbar[j] += g * u[n][i] * A[4 * i + j];
            }
        for (int k = n; k >= 1; --k) {
            /* v^(k) = 1 / b,  b = A^T u^(k):  bbar = -vbar v^2 */
            double bbar[4];
            for (int j = 0; j < 4; ++j) bbar[j] = -vbar[j] * v[k][j] * v[k][j];
            for (int i = 0; i < 4; ++i)
                for (int j = 0; j < 4; ++j) {
                    ubar[i] += A[4 * i + j] * bbar[j];
                    Abar[4 * i + j] += u[k][i] * bbar[j];
                }
            /* u^(k) = 1 / a,  a = A v^(k-1):  abar = -ubar u^2 */
            double abar[4];
            for (int i = 0; i < 4; ++i) abar[i] = -ubar[i] * u[k][i] * u[k][i];
            for (int j = 0; j < 4; ++j) vbar[j] = 0.0;
            for (int i = 0; i < 4; ++i)
                for (int j = 0; j < 4; ++j) {
                    vbar[j] += A[4 * i + j] * abar[i];
                    Abar[4 * i + j] += abar[i] * v[k - 1][j];
                }
            for (int i = 0; i < 4; ++i) ubar[i] = 0.0;
        }
        for (int q = 0; q < 16; ++q) dH[16 * b + q] = Abar[q] * A[q];
    }
    return 0;
}

int oracle_version(void) { return 1; }
