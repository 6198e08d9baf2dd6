"""Pins for the size-generic fp64 oracle (n x n Birkhoff projection), CPU only.

Independent routes to what the paper fixes for every n: the 4 x 4 oracle (a separate
implementation) at n = 4; Sinkhorn-Knopp run to convergence (eq. sinkhorn_knopp, a
different algorithm for the same projection); doubly stochastic output with
log P - H = alpha_i + beta_j (eq. dual, primal recovery); the uniform matrix for
additively separable H; equivariance under row and column permutations; and for
the backward, central finite differences of the forward, the Jacobian of the
linearised optimality conditions, and the closed form at separable H.
"""
import numpy as np
import pytest

import oracle
from oracle import birkhoffn as on


def gauss(B, n, sigma, seed):
    rng = np.random.default_rng(seed)
    return sigma * rng.standard_normal((B, n, n)), rng.standard_normal((B, n, n))


def near_permutation(B, n, gap, noise, seed):
    rng = np.random.default_rng(seed)
    H = noise * rng.standard_normal((B, n, n))
    for b in range(B):
        H[b, np.arange(n), rng.permutation(n)] += gap
    return H


def _proj(H, tol=1e-14):
    P, dual, it = on.fwd(H, tol=tol)
    assert (it >= 0).all()
    return P


@pytest.mark.parametrize("sigma", [0.5, 5.0, 20.0])
def test_matches_4x4_oracle(sigma):
    H, G = gauss(3000, 4, sigma, seed=1)
    P4, d4, it4 = oracle.fwd(H)
    P, d, it = on.fwd(H)
    # the two take the same steps up to rounding, which can move the last one across tol
    assert (it == it4).mean() > 0.999 and np.abs(it - it4).max() <= 1
    assert np.abs(P - P4).max() < 1e-13
    if sigma <= 5.0:  # at larger logits the dual is ill-determined in finite precision
        assert np.abs(d - d4).max() < 1e-10
    assert np.abs(on.bwd(P, G) - oracle.bwd(P4, G)).max() < 1e-12


def test_matches_4x4_oracle_near_permutations():
    H = near_permutation(2000, 4, 20.0, 0.1, seed=2)
    G = np.random.default_rng(3).standard_normal(H.shape)
    P4, _, _ = oracle.fwd(H)
    P, _, _ = on.fwd(H)
    assert np.abs(P - P4).max() < 1e-13
    assert np.abs(on.bwd(P, G) - oracle.bwd(P4, G)).max() < 1e-12


@pytest.mark.parametrize("n,sigma", [(3, 2.0), (5, 5.0), (8, 1.0), (8, 5.0), (16, 3.0)])
def test_matches_sinkhorn(n, sigma):
    H, _ = gauss(300, n, sigma, seed=4 + n)
    P = _proj(H)
    Ps, steps = on.sinkhorn(H, tol=1e-15, max_steps=400000)
    ok = steps < 400000  # Sinkhorn is slow where the problem is badly scaled
    assert ok.mean() > 0.9
    assert np.abs(P[ok] - Ps[ok]).max() < 1e-12


@pytest.mark.parametrize("n,sigma", [(2, 3.0), (6, 10.0), (8, 1.0), (8, 20.0), (8, 50.0), (12, 10.0)])
def test_doubly_stochastic_and_dual(n, sigma):
    H, _ = gauss(500, n, sigma, seed=10 + n)
    P, dual, it = on.fwd(H)
    assert (it >= 0).all()
    assert on.marginal_errors(P).max() < 1e-12
    alpha, beta = dual[:, :n], dual[:, n:]
    assert (beta[:, -1] == 0).all()
    big = P > 1e-200
    resid = np.log(np.where(big, P, 1.0)) - H - alpha[:, :, None] - beta[:, None, :]
    assert np.abs(np.where(big, resid, 0.0)).max() < 1e-9 * max(1.0, sigma)


@pytest.mark.parametrize("n", [3, 8, 16])
def test_separable_gives_uniform(n):
    rng = np.random.default_rng(20 + n)
    u = 10 * rng.standard_normal((100, n, 1))
    v = 10 * rng.standard_normal((100, 1, n))
    P, dual, it = on.fwd(u + v)
    assert (it >= 0).all()
    assert np.abs(P - 1.0 / n).max() < 1e-13
    # alpha_i + beta_j = log(1/n) - u_i - v_j
    s = dual[:, :n, None] + dual[:, None, n:]
    assert np.abs(s - (np.log(1.0 / n) - u - v)).max() < 1e-9


@pytest.mark.parametrize("n", [5, 8])
def test_permutation_equivariance(n):
    rng = np.random.default_rng(30 + n)
    H, G = gauss(200, n, 6.0, seed=31)
    pr, pc = rng.permutation(n), rng.permutation(n)
    P = _proj(H)
    Pp = _proj(H[:, pr][:, :, pc])
    assert np.abs(Pp - P[:, pr][:, :, pc]).max() < 1e-13
    dH = on.bwd(P, G)
    dHp = on.bwd(Pp, G[:, pr][:, :, pc])
    assert np.abs(dHp - dH[:, pr][:, :, pc]).max() < 1e-11


def test_near_permutations_n8():
    H = near_permutation(1000, 8, 20.0, 0.1, seed=40)
    P, _, it = on.fwd(H)
    assert (it >= 0).all()
    assert on.marginal_errors(P).max() < 1e-12


def test_non_finite_input():
    H, _ = gauss(4, 8, 1.0, seed=41)
    H[2, 3, 5] = np.nan
    P, dual, it = on.fwd(H)
    assert list(it[[0, 1, 3]] >= 0) == [True] * 3 and it[2] == -2
    assert np.isnan(P[2]).all() and np.isnan(dual[2]).all()
    assert np.isfinite(P[[0, 1, 3]]).all()


@pytest.mark.parametrize("n,sigma", [(3, 1.0), (8, 0.5), (8, 3.0), (8, 10.0)])
def test_backward_finite_differences(n, sigma):
    H, G = gauss(4, n, sigma, seed=50 + n)
    P = _proj(H)
    dH = on.bwd(P, G)
    h = 1e-5
    fd = np.zeros_like(H)
    for k in range(n):
        for l in range(n):
            E = np.zeros((n, n))
            E[k, l] = h
            fd[:, k, l] = (G * (_proj(H + E) - _proj(H - E))).sum(axis=(1, 2)) / (2 * h)
    scale = np.maximum(1.0, np.abs(fd).max(axis=(1, 2)))
    assert (np.abs(dH - fd).max(axis=(1, 2)) / scale).max() < 2e-7


def kkt_jacobian(P):
    """J[b, n i + j, n k + l] = dP_ij / dH_kl from the linearised conditions
    delta P = P o (delta H + delta alpha 1^T + 1 delta beta^T), zero changes of the
    row sums and of the first n - 1 column sums, delta beta_n = 0."""
    B, n = P.shape[0], P.shape[1]
    r, c = P.sum(axis=2), P.sum(axis=1)
    M = np.zeros((B, 2 * n - 1, 2 * n - 1))
    M[:, range(n), range(n)] = r
    M[:, :n, n:] = P[:, :, : n - 1]
    M[:, n:, :n] = np.transpose(P[:, :, : n - 1], (0, 2, 1))
    M[:, range(n, 2 * n - 1), range(n, 2 * n - 1)] = c[:, : n - 1]
    J = np.zeros((B, n * n, n * n))
    for kl in range(n * n):
        E = np.zeros((n, n))
        E.flat[kl] = 1.0
        PE = P * E
        rhs = -np.concatenate([PE.sum(axis=2), PE.sum(axis=1)[:, : n - 1]], axis=1)
        sol = np.linalg.solve(M, rhs[..., None])[..., 0]
        db = np.concatenate([sol[:, n:], np.zeros((B, 1))], axis=1)
        J[:, :, kl] = (P * (E[None] + sol[:, :n, None] + db[:, None, :])).reshape(B, n * n)
    return J


@pytest.mark.parametrize("n,sigma", [(5, 2.0), (8, 1.0), (8, 6.0)])
def test_backward_kkt_jacobian(n, sigma):
    H, G = gauss(100, n, sigma, seed=60 + n)
    P = _proj(H)
    vjp = np.einsum("bij,bi->bj", kkt_jacobian(P), G.reshape(-1, n * n)).reshape(-1, n, n)
    assert np.abs(on.bwd(P, G) - vjp).max() < 1e-10


@pytest.mark.parametrize("n", [3, 8])
def test_backward_separable_closed_form(n):
    # at P = J/n the projection's Jacobian is (1/n) times double centring
    rng = np.random.default_rng(70 + n)
    H = 4 * rng.standard_normal((50, n, 1)) + 4 * rng.standard_normal((50, 1, n))
    G = rng.standard_normal((50, n, n))
    C = np.eye(n) - 1.0 / n
    assert np.abs(on.bwd(_proj(H), G) - (C @ G @ C) / n).max() < 1e-13


@pytest.mark.parametrize("n,sigma", [(8, 2.0), (8, 30.0)])
def test_backward_row_and_column_sums_vanish(n, sigma):
    # P is unchanged by adding a constant to a row or column of H
    H, G = gauss(400, n, sigma, seed=80 + n)
    dH = on.bwd(_proj(H), G)
    scale = np.maximum(1.0, np.abs(dH).max(axis=(1, 2)))
    assert (np.abs(dH.sum(axis=2)).max(axis=1) / scale).max() < 1e-10
    assert (np.abs(dH.sum(axis=1)).max(axis=1) / scale).max() < 1e-10
