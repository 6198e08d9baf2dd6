"""Pins for the general entropic-OT oracle (cost M, marginals a, b, regulariser eta), CPU only.

Routes that the paper fixes independently of the oracle's Newton iteration: the Birkhoff
projection as the special case M = -H, eta = 1, a = b = 1 (Sec. 2.3); Sinkhorn's scaling
iteration with marginals (eq. sinkhorn_knopp generalised as in Sec. 2.3: u = a / (K v),
v = b / (K^T u)); the marginal constraints and primal recovery T_ij = exp((alpha_i + beta_j -
M_ij) / eta) (eq. dual); the product coupling a b^T / sum(a) for additively separable M; the
scaling T(M, eta) = T(M / eta, 1); and for the backward (eq. derivative) central finite
differences, the closed form at separable M, and invariance to row and column shifts of M.
"""
import numpy as np
import pytest

from oracle import birkhoffn as on


def problem(B, n, scale, seed, eta_ok=True):
    rng = np.random.default_rng(seed)
    M = scale * rng.standard_normal((B, n, n))
    a = rng.uniform(0.2, 2.0, (B, n))
    b = rng.uniform(0.2, 2.0, (B, n))
    b *= (a.sum(1) / b.sum(1))[:, None]
    G = rng.standard_normal((B, n, n))
    return M, a, b, G


def _ot(M, a, b, eta, tol=1e-14):
    T, dual, it = on.ot_fwd(M, a, b, eta, tol=tol)
    assert (it >= 0).all()
    return T, dual


@pytest.mark.parametrize("n", [4, 8])
def test_birkhoff_special_case(n):
    rng = np.random.default_rng(n)
    H = 5 * rng.standard_normal((500, n, n))
    G = rng.standard_normal(H.shape)
    P, d, _ = on.fwd(H)
    ones = np.ones((500, n))
    T, dual, it = on.ot_fwd(-H, ones, ones, 1.0)
    assert (it >= 0).all()
    assert np.abs(T - P).max() < 1e-14
    assert np.abs(dual - d).max() < 1e-10
    # dL/dM = -dL/dH for M = -H
    assert np.abs(on.ot_bwd(T, ones, G, 1.0) + on.bwd(P, G)).max() < 1e-13


@pytest.mark.parametrize("n,eta,scale", [(4, 1.0, 3.0), (4, 0.2, 3.0), (4, 4.0, 10.0), (6, 0.5, 2.0), (8, 1.0, 2.0)])
def test_matches_sinkhorn_with_marginals(n, eta, scale):
    M, a, b, _ = problem(300, n, scale, seed=int(10 * eta) + n)
    T, _ = _ot(M, a, b, eta)
    Ts, steps = on.ot_sinkhorn(M, a, b, eta, tol=1e-15, max_steps=400000)
    ok = steps < 400000
    assert ok.mean() > 0.9
    assert np.abs(T[ok] - Ts[ok]).max() < 1e-12


@pytest.mark.parametrize("n,eta,scale", [(3, 1.0, 5.0), (4, 0.05, 2.0), (4, 1.0, 30.0), (8, 0.5, 5.0)])
def test_marginals_and_primal_recovery(n, eta, scale):
    M, a, b, _ = problem(400, n, scale, seed=20 + n)
    T, dual = _ot(M, a, b, eta)
    assert np.abs(T.sum(2) - a).max() < 1e-12
    assert np.abs(T.sum(1) - b).max() < 1e-12
    assert (dual[:, -1] == 0).all()
    big = T > 1e-200
    resid = eta * np.log(np.where(big, T, 1.0)) - (dual[:, :n, None] + dual[:, None, n:] - M)
    assert np.abs(np.where(big, resid, 0.0)).max() < 1e-9 * max(1.0, scale)


@pytest.mark.parametrize("n,eta", [(4, 0.3), (8, 2.0)])
def test_separable_cost_gives_product_coupling(n, eta):
    rng = np.random.default_rng(30 + n)
    B = 100
    M = 4 * rng.standard_normal((B, n, 1)) + 4 * rng.standard_normal((B, 1, n))
    a = rng.uniform(0.5, 3.0, (B, n))
    b = rng.uniform(0.5, 3.0, (B, n))
    b *= (a.sum(1) / b.sum(1))[:, None]
    T, _ = _ot(M, a, b, eta)
    expect = a[:, :, None] * b[:, None, :] / a.sum(1)[:, None, None]
    assert np.abs(T - expect).max() < 1e-13


@pytest.mark.parametrize("eta", [0.1, 2.5])
def test_regulariser_scaling(eta):
    M, a, b, _ = problem(300, 4, 2.0, seed=40)
    T1, d1 = _ot(M, a, b, eta)
    T2, d2 = _ot(M / eta, a, b, 1.0)
    assert np.abs(T1 - T2).max() < 1e-13
    assert np.abs(d1 - eta * d2).max() < 1e-9


def test_permutation_equivariance():
    M, a, b, G = problem(200, 5, 3.0, seed=50)
    rng = np.random.default_rng(51)
    pr, pc = rng.permutation(5), rng.permutation(5)
    T, _ = _ot(M, a, b, 0.7)
    Tp, _ = _ot(M[:, pr][:, :, pc], a[:, pr], b[:, pc], 0.7)
    assert np.abs(Tp - T[:, pr][:, :, pc]).max() < 1e-13
    dM = on.ot_bwd(T, a, G, 0.7)
    dMp = on.ot_bwd(Tp, a[:, pr], G[:, pr][:, :, pc], 0.7)
    assert np.abs(dMp - dM[:, pr][:, :, pc]).max() < 1e-11


@pytest.mark.parametrize("n,eta,scale", [(3, 1.0, 1.0), (4, 0.5, 2.0), (4, 2.0, 5.0), (8, 1.0, 1.0)])
def test_backward_finite_differences(n, eta, scale):
    M, a, b, G = problem(4, n, scale, seed=60 + n)
    T, _ = _ot(M, a, b, eta)
    dM = on.ot_bwd(T, a, G, eta)
    h = 1e-5
    fd = np.zeros_like(M)
    for k in range(n):
        for l in range(n):
            E = np.zeros((n, n))
            E[k, l] = h
            Tp, _ = _ot(M + E, a, b, eta)
            Tm, _ = _ot(M - E, a, b, eta)
            fd[:, k, l] = (G * (Tp - Tm)).sum(axis=(1, 2)) / (2 * h)
    scale_ = np.maximum(1.0, np.abs(fd).max(axis=(1, 2)))
    assert (np.abs(dM - fd).max(axis=(1, 2)) / scale_).max() < 2e-7


@pytest.mark.parametrize("n,eta", [(4, 0.5), (6, 1.5)])
def test_backward_separable_closed_form(n, eta):
    # at T = a b^T / s the linearised conditions give dT = -(T / eta) o C(dM), C the centring
    # X - X b 1^T / s - 1 a^T X / s + (a^T X b) / s^2; so dL/dM = -(1/eta) C*(G o T)
    rng = np.random.default_rng(70 + n)
    B = 50
    M = 3 * rng.standard_normal((B, n, 1)) + 3 * rng.standard_normal((B, 1, n))
    a = rng.uniform(0.5, 2.0, (B, n))
    b = rng.uniform(0.5, 2.0, (B, n))
    b *= (a.sum(1) / b.sum(1))[:, None]
    G = rng.standard_normal((B, n, n))
    T, _ = _ot(M, a, b, eta)
    s = a.sum(1)[:, None, None]
    Y = G * T
    r = Y.sum(2, keepdims=True)
    c = Y.sum(1, keepdims=True)
    tot = Y.sum((1, 2), keepdims=True)
    Cstar = Y - b[:, None, :] * r / s - a[:, :, None] * c / s + a[:, :, None] * b[:, None, :] * tot / s ** 2
    assert np.abs(on.ot_bwd(T, a, G, eta) + Cstar / eta).max() < 1e-13


def test_backward_row_and_column_sums_vanish():
    # T is unchanged by adding a constant to a row or a column of M
    M, a, b, G = problem(300, 4, 10.0, seed=80)
    T, _ = _ot(M, a, b, 0.8)
    dM = on.ot_bwd(T, a, G, 0.8)
    scale = np.maximum(1.0, np.abs(dM).max(axis=(1, 2)))
    assert (np.abs(dM.sum(axis=2)).max(axis=1) / scale).max() < 1e-10
    assert (np.abs(dM.sum(axis=1)).max(axis=1) / scale).max() < 1e-10
