"""Independent reference routes used to pin the oracle (test helpers only).

Nothing here calls the oracle or the HIP path. Each helper is a different
route to a quantity the paper fixes:

* ``planted``: inputs whose projection is known exactly, built from the
  Birkhoff-von Neumann form and the uniqueness of the Sinkhorn scaling (Sec. 2.2);
* ``log_sinkhorn``: block-coordinate ascent (eq. bca) in the log domain, run
  until the marginals are exact to ~1e-14;
* ``kkt_jacobian``: dP/dH from linearising P_ij = exp(H_ij + alpha_i + beta_j)
  with fixed marginals (the KKT system behind eq. dual), solved by numpy;
* ``literal_*_decimal``: the paper's own 4x4 formulas written literally (Sec. 3.2
  Hessian diag(c) - T^T T with Cramer's rule eq. newton_direction; eq. derivative
  for the backward) in high-precision decimal arithmetic, where their
  cancellations are harmless.
"""
from __future__ import annotations

import decimal
from decimal import Decimal

import numpy as np

from workloads import PERMS4


# ---------------------------------------------------------------------------
# Planted solutions
# ---------------------------------------------------------------------------
def planted(B: int, sigma: float, seed: int, shift_scale: float = 3.0):
    """H = log P0 + a 1^T + 1 b^T with P0 = sum_k lam_k Pi_k / sum_k lam_k.

    P0 is in the interior of the Birkhoff polytope (Birkhoff-von Neumann), so by
    uniqueness of the scaling the projection of exp(H) is exactly P0, with
    beta_j = b_4 - b_j and alpha_i = -a_i - b_4 under the gauge beta_4 = 0.
    """
    rng = np.random.default_rng(np.random.SeedSequence([seed, 77, int(sigma * 100)]))
    z = rng.standard_normal((B, 24))
    lam = np.exp(sigma * (z - z.max(axis=1, keepdims=True)))
    lam /= lam.sum(axis=1, keepdims=True)
    P0 = np.zeros((B, 4, 4))
    rows = np.arange(4)
    for k in range(24):
        P0[:, rows, PERMS4[k]] += lam[:, k:k + 1]
    a = shift_scale * rng.standard_normal((B, 4))
    b = shift_scale * rng.standard_normal((B, 4))
    H = np.log(P0) + a[:, :, None] + b[:, None, :]
    alpha = -a - b[:, 3:4]
    beta = b[:, 3:4] - b
    return H, P0, alpha, beta


# ---------------------------------------------------------------------------
# Log-domain block-coordinate ascent (Sinkhorn-Knopp) to convergence
# ---------------------------------------------------------------------------
def _lse(x, axis):
    m = x.max(axis=axis, keepdims=True)
    return (m + np.log(np.exp(x - m).sum(axis=axis, keepdims=True))).squeeze(axis)


def log_sinkhorn(H, tol: float = 1e-14, max_iter: int = 200000):
    H = np.asarray(H, np.float64)
    beta = np.zeros(H.shape[:-2] + (4,))
    for _ in range(max_iter):
        alpha = -_lse(H + beta[..., None, :], axis=-1)
        beta = -_lse(H + alpha[..., :, None], axis=-2)
        P = np.exp(H + alpha[..., :, None] + beta[..., None, :])
        err = np.abs(P.sum(axis=-1) - 1).max()
        if err <= tol:
            return P
    raise RuntimeError("log-domain Sinkhorn did not converge")


# ---------------------------------------------------------------------------
# KKT-linearisation Jacobian
# ---------------------------------------------------------------------------
def kkt_jacobian(P):
    """J[b, 4i+j, 4k+l] = dP_ij / dH_kl at the doubly stochastic P[b].

    delta P_ij = P_ij (delta H_ij + delta alpha_i + delta beta_j) with zero
    changes of all row sums and of the first three column sums, delta beta_4 = 0.
    """
    P = np.asarray(P, np.float64)
    B = P.shape[0]
    J = np.zeros((B, 16, 16))
    r = P.sum(axis=2)
    c = P.sum(axis=1)
    M = np.zeros((B, 7, 7))
    M[:, range(4), range(4)] = r
    M[:, :4, 4:] = P[:, :, :3]
    M[:, 4:, :4] = np.transpose(P[:, :, :3], (0, 2, 1))
    M[:, range(4, 7), range(4, 7)] = c[:, :3]
    for kl in range(16):
        k, l = divmod(kl, 4)
        E = np.zeros((4, 4))
        E[k, l] = 1.0
        PE = P * E
        rhs = -np.concatenate([PE.sum(axis=2), PE.sum(axis=1)[:, :3]], axis=1)
        sol = np.linalg.solve(M, rhs[..., None])[..., 0]
        da = sol[:, :4]
        db = np.concatenate([sol[:, 4:], np.zeros((B, 1))], axis=1)
        dP = P * (E[None] + da[:, :, None] + db[:, None, :])
        J[:, :, kl] = dP.reshape(B, 16)
    return J


# ---------------------------------------------------------------------------
# The paper's literal 4x4 formulas in decimal arithmetic
# ---------------------------------------------------------------------------
def _dec_matrix(x):
    return [[Decimal(float(x[i][j])) for j in range(4)] for i in range(4)]


def _row_softmax_dec(H, beta):
    T = [[None] * 4 for _ in range(4)]
    lse = [None] * 4
    for i in range(4):
        U = [beta[j] + H[i][j] for j in range(4)]
        mu = max(U)
        e = [(u - mu).exp() for u in U]
        s = sum(e)
        for j in range(4):
            T[i][j] = e[j] / s
        lse[i] = mu + s.ln()
    return T, lse


def _cramer3(h, g):
    """d = -h^{-1} g by eq. newton_direction (adjugate / determinant)."""
    h11, h12, h13 = h[0]
    h22, h23 = h[1][1], h[1][2]
    h33 = h[2][2]
    g1, g2, g3 = g
    det = (h11 * (h22 * h33 - h23 * h23) - h12 * (h12 * h33 - h23 * h13)
           + h13 * (h12 * h23 - h22 * h13))
    d1 = -((h22 * h33 - h23 * h23) * g1 + (h13 * h23 - h12 * h33) * g2
           + (h12 * h23 - h22 * h13) * g3) / det
    d2 = -((h13 * h23 - h12 * h33) * g1 + (h11 * h33 - h13 * h13) * g2
           + (h12 * h13 - h11 * h23) * g3) / det
    d3 = -((h12 * h23 - h22 * h13) * g1 + (h12 * h13 - h11 * h23) * g2
           + (h11 * h22 - h12 * h12) * g3) / det
    return [d1, d2, d3]


def literal_newton_decimal(H, beta0=None, prec: int = 100, tol_exp: int = 60,
                           max_iter: int = 400, full: bool = False):
    """Newton on f (Sec. 3.1) with the literal 4x4 gradient/Hessian (Sec. 3.2).

    Armijo halving on f, in ``prec``-digit decimal arithmetic; returns T* (as
    Decimals) once every column sum is within 10^-tol_exp of one, and with
    ``full`` also beta (beta_4 = 0) and the row log-sum-exps lse_i, so that
    alpha_i = -lse_i (eq. alpha_opt with unit rows).
    """
    with decimal.localcontext() as ctx:
        ctx.prec = prec
        Hd = _dec_matrix(H)
        beta = [Decimal(0)] * 4 if beta0 is None else [Decimal(float(x)) for x in beta0]
        beta[3] = Decimal(0)
        tol = Decimal(10) ** (-tol_exp)
        for _ in range(max_iter):
            T, lse = _row_softmax_dec(Hd, beta)
            c = [sum(T[i][j] for i in range(4)) for j in range(4)]
            if max(abs(cj - 1) for cj in c) <= tol:
                return (T, beta, lse) if full else T
            g = [c[j] - 1 for j in range(3)]
            # h = diag(c) - T_{-m}^T T_{-m}   (Sec. 3.2)
            h = [[(c[j] if j == k else Decimal(0)) - sum(T[i][j] * T[i][k] for i in range(4))
                  for k in range(3)] for j in range(3)]
            d = _cramer3(h, g)
            f0 = sum(lse) - sum(beta[:3])
            slope = sum(g[j] * d[j] for j in range(3))
            t = Decimal(1)
            for _ in range(200):
                bn = [beta[j] + t * d[j] for j in range(3)] + [Decimal(0)]
                _, ln = _row_softmax_dec(Hd, bn)
                if sum(ln) - sum(bn[:3]) <= f0 + Decimal("1e-4") * t * slope:
                    break
                t /= 2
            beta = bn
        raise RuntimeError("literal Newton did not converge")


def literal_backward_decimal(T, G, prec: int = 100):
    """eq. derivative with eta = 1, a = b = 1, m = 4, literally; returns dH = -D."""
    with decimal.localcontext() as ctx:
        ctx.prec = prec
        Gd = _dec_matrix(G)
        Gam = [[Gd[i][j] * T[i][j] for j in range(4)] for i in range(4)]
        mu_r = [sum(Gam[i]) for i in range(4)]
        mu_c = [sum(Gam[i][j] for i in range(4)) for j in range(3)]
        # Delta = diag(b_{-m}) - T_{-m}^T T_{-m}
        Delta = [[(Decimal(1) if j == k else Decimal(0)) - sum(T[i][j] * T[i][k] for i in range(4))
                  for k in range(3)] for j in range(3)]
        rhs = [mu_c[j] - sum(T[i][j] * mu_r[i] for i in range(4)) for j in range(3)]
        # Cramer's rule returns -Delta^{-1} rhs
        wm = [-x for x in _cramer3(Delta, rhs)]
        w = wm + [Decimal(0)]
        v = [mu_r[i] - sum(T[i][j] * w[j] for j in range(3)) for i in range(4)]
        D = [[(v[i] + w[j] - Gd[i][j]) * T[i][j] for j in range(4)] for i in range(4)]
        return np.array([[-float(D[i][j]) for j in range(4)] for i in range(4)])


def dec_to_float(T):
    return np.array([[float(T[i][j]) for j in range(4)] for i in range(4)])
