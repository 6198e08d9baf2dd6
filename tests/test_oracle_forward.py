"""Pins for the oracle's forward projection (CPU only).

Each check comes from something the paper fixes, not from the oracle's own
formulas: planted solutions and closed forms (uniqueness of the Sinkhorn scaling,
Sec. 2.2), the KKT form of the solution (eq. dual), invariances, agreement with
block-coordinate ascent run to convergence (eq. bca), and the paper's literal
4x4 Newton formulas in high precision (Sec. 3.2).
"""
import numpy as np
import pytest

import oracle
import workloads
from tests import _refs


def _fwd(H, **kw):
    P, dual, it = oracle.fwd(H, **kw)
    assert (it >= 0).all(), "oracle did not converge"
    return P, dual, it


@pytest.mark.parametrize("sigma", [0.3, 2.0, 8.0, 20.0])
def test_planted_solution(sigma):
    H, P0, alpha, beta = _refs.planted(400, sigma, seed=1)
    P, dual, _ = _fwd(H)
    assert np.abs(P - P0).max() < 1e-12
    # the dual is pinned too wherever the problem is well conditioned
    ok = P0.min(axis=(1, 2)) > 1e-6
    assert ok.sum() >= 5
    assert np.abs(dual[ok, :4] - alpha[ok]).max() < 1e-8
    assert np.abs(dual[ok, 4:] - beta[ok]).max() < 1e-8
    assert (dual[:, 7] == 0).all()


def test_planted_near_permutation():
    # lam spread of e^{20 * 5} -> entries as small as ~1e-40: the hard regime
    H, P0, _, _ = _refs.planted(200, 60.0, seed=2)
    P, _, _ = _fwd(H)
    assert P0.min() < 1e-20
    assert np.abs(P - P0).max() < 1e-12


def test_separable_gives_uniform():
    rng = np.random.default_rng(3)
    a = 20 * rng.standard_normal((100, 4, 1))
    b = 20 * rng.standard_normal((100, 1, 4))
    P, dual, it = _fwd(a + b)
    assert np.abs(P - 0.25).max() < 1e-13


def test_latin_square_closed_form():
    # Every row and column of exp(H) holds each e^{v_k} once: exp(H)/sum_k e^{v_k}
    # is already doubly stochastic, hence the projection.
    rng = np.random.default_rng(4)
    L = np.array([[0, 1, 2, 3], [1, 0, 3, 2], [2, 3, 0, 1], [3, 2, 1, 0]])
    for _ in range(20):
        v = 6 * rng.standard_normal(4)
        pr = rng.permutation(4)
        pc = rng.permutation(4)
        H = v[L][pr][:, pc] + rng.standard_normal((4, 1)) * 5 + rng.standard_normal((1, 4)) * 5
        P, _, _ = _fwd(H[None])
        expect = np.exp(v[L][pr][:, pc]) / np.exp(v).sum()
        assert np.abs(P[0] - expect).max() < 1e-13


def test_scaled_permutation_closed_form():
    # H = t Pi: P = (J + (e^t - 1) Pi) / (e^t + 3)
    for t in [0.5, 3.0, 15.0]:
        for k in [0, 7, 23]:
            Pi = np.zeros((4, 4))
            Pi[np.arange(4), workloads.PERMS4[k]] = 1
            P, _, _ = _fwd(t * Pi[None])
            expect = (np.ones((4, 4)) + np.expm1(t) * Pi) / (np.exp(t) + 3)
            assert np.abs(P[0] - expect).max() < 1e-13


def test_kronecker_closed_form():
    # H = J_2 (x) h: P = 1/2 J_2 (x) Q, Q_11 = 1/(1 + exp(-s/2)), s = h11 + h22 - h12 - h21
    rng = np.random.default_rng(5)
    for _ in range(20):
        h = 8 * rng.standard_normal((2, 2))
        H = np.kron(np.ones((2, 2)), h)
        P, _, _ = _fwd(H[None])
        s = h[0, 0] + h[1, 1] - h[0, 1] - h[1, 0]
        q = 1 / (1 + np.exp(-s / 2))
        Q = np.array([[q, 1 - q], [1 - q, q]])
        assert np.abs(P[0] - 0.5 * np.kron(np.ones((2, 2)), Q)).max() < 1e-13


@pytest.mark.parametrize("sigma", [1.0, 10.0, 50.0])
def test_kkt_certificate(sigma):
    H, _ = workloads.gauss(2000, sigma, seed=6)
    H = H.astype(np.float64)
    P, dual, _ = _fwd(H)
    linf, _ = oracle.marginal_errors(P)
    assert linf.max() <= 1.5e-13
    assert (P >= 0).all()
    # log P - H = alpha_i + beta_j exactly (eq. dual), beta_4 = 0
    logP = np.log(np.maximum(P, 1e-300))
    kkt = logP - H - dual[:, :4, None] - dual[:, None, 4:]
    mask = P > 1e-290
    assert np.abs(kkt[mask]).max() < 1e-11 * max(1.0, sigma)
    assert (dual[:, 7] == 0).all()


def test_invariances():
    rng = np.random.default_rng(7)
    H = 10 * rng.standard_normal((300, 4, 4))
    P, _, _ = _fwd(H)
    # additive row/column shifts (Sec. 3.1: the dual has this redundancy)
    Hs = H + 7 * rng.standard_normal((300, 4, 1)) + 7 * rng.standard_normal((300, 1, 4))
    Ps, _, _ = _fwd(Hs)
    assert np.abs(Ps - P).max() < 1e-12
    # row/column permutation equivariance and transposition
    pr, pc = rng.permutation(4), rng.permutation(4)
    Pp, _, _ = _fwd(H[:, pr][:, :, pc])
    assert np.abs(Pp - P[:, pr][:, :, pc]).max() < 1e-12
    Pt, _, _ = _fwd(np.transpose(H, (0, 2, 1)))
    assert np.abs(Pt - np.transpose(P, (0, 2, 1))).max() < 1e-12


def test_fixed_point():
    H, P0, _, _ = _refs.planted(100, 2.0, seed=8, shift_scale=0.0)
    P, _, _ = _fwd(np.log(P0))
    assert np.abs(P - P0).max() < 1e-13


@pytest.mark.parametrize("sigma", [0.1, 1.0, 2.0])
def test_agrees_with_converged_sinkhorn(sigma):
    H, _ = workloads.gauss(500, sigma, seed=9)
    H = H.astype(np.float64)
    P, _, _ = _fwd(H)
    Psk = _refs.log_sinkhorn(H, tol=1e-14)
    assert np.abs(P - Psk).max() < 1e-12


@pytest.mark.parametrize("sigma,prec", [(5.0, 60), (20.0, 80), (50.0, 120)])
def test_literal_formulas_high_precision(sigma, prec):
    """The paper's literal Hessian diag(c) - T^T T and Cramer's rule, in
    prec-digit decimals, polish to the same P as the oracle's rearranged
    fp64 forms."""
    H, _ = workloads.gauss(6, sigma, seed=10)
    H = H.astype(np.float64)
    P, dual, _ = _fwd(H)
    for b in range(H.shape[0]):
        T = _refs.literal_newton_decimal(H[b], beta0=dual[b, 4:], prec=prec,
                                         tol_exp=prec // 2)
        assert np.abs(_refs.dec_to_float(T) - P[b]).max() < 1e-13


def test_stop_rule_and_iteration_report():
    H, _ = workloads.gauss(200, 5.0, seed=11)
    H = H.astype(np.float64)
    P, dual, it = oracle.fwd(H, tol=1e-13, max_iter=0)
    # max_iter = 0 returns T(x^(0)) = row softmax of H, flagged unconverged
    rs = np.exp(H - H.max(axis=2, keepdims=True))
    rs /= rs.sum(axis=2, keepdims=True)
    assert np.abs(P - rs).max() < 1e-15
    assert (it == -1).all()
    P2, _, it2 = oracle.fwd(H, tol=1e-3)
    linf, _ = oracle.marginal_errors(P2)
    assert (it2 >= 0).all() and linf.max() <= 1.01e-3


def test_non_finite_input():
    H = np.zeros((3, 4, 4))
    H[1, 2, 3] = np.nan
    H[2, 0, 0] = np.inf
    P, dual, it = oracle.fwd(H)
    assert list(it) == [0, -2, -2]
    assert np.isnan(P[1]).all() and np.isnan(P[2]).all()
    assert np.abs(P[0] - 0.25).max() == 0.0


def test_workload_samples_converge():
    for name in ["mix_bf16_b2e24", "logunif_b2e25"]:
        ch = workloads.make_chunk(workloads.WORKLOADS[name], 3, B=3 * workloads.CHUNK + 20000)
        P, dual, it = oracle.fwd(ch.H)
        assert (it >= 0).all()
        assert oracle.marginal_errors(P)[0].max() <= 1.5e-13


def _lap_inv_norm(P: np.ndarray) -> float:
    """|L^-1|_inf of the reduced dual's Hessian at P: the Laplacian of the column graph
    with weights sum_i P_ij P_ik, grounded at column 4. A column-sum residual r moves the
    potentials by at most this times |r|_inf (to first order)."""
    W = P.T @ P
    np.fill_diagonal(W, 0.0)
    L = -W[:3, :3]
    L[np.arange(3), np.arange(3)] = W[:3].sum(axis=1)
    with np.errstate(all="ignore"):
        n = np.abs(np.linalg.inv(L)).sum(axis=1).max()
    return float(n) if np.isfinite(n) else np.inf


LITERAL_FAMILIES = [("gauss", 0.3), ("gauss", 1.0), ("gauss", 5.0), ("gauss", 20.0), ("gauss", 50.0),
                    ("uniform", 1.0), ("uniform", 10.0)]


@pytest.mark.parametrize("family,scale", LITERAL_FAMILIES)
def test_literal_newton_from_zero(family, scale):
    """The paper's literal Newton (Hessian diag(c) - T^T T, Cramer's rule, Armijo
    halving) in decimals, started at beta = 0 and not at the oracle's solution,
    reaches the oracle's P, and its dual (alpha = -lse, beta with beta_4 = 0) wherever
    the conditioning of the reduced Hessian lets fp64 determine it."""
    prec = 60 if scale <= 5 else (80 if scale <= 20 else 120)
    gen = workloads.gauss if family == "gauss" else workloads.uniform
    H, _ = gen(10, scale, seed=12, grad=False)
    H = H.astype(np.float64)
    P, dual, it = _fwd(H)
    assert (it >= 0).all()
    for b in range(H.shape[0]):
        T, beta, lse = _refs.literal_newton_decimal(H[b], prec=prec, tol_exp=prec // 2, full=True)
        Tf = _refs.dec_to_float(T)
        assert np.abs(Tf - P[b]).max() < 1e-13
        ref = np.array([-float(x) for x in lse] + [float(x) for x in beta])
        assert ref[7] == 0.0 and dual[b, 7] == 0.0
        # the oracle stops at column residual 1e-13; fp64 rounding of the sums adds ~1e-15
        bound = 2.0 * _lap_inv_norm(Tf) * 1e-13 + 1e-13 * (1.0 + np.abs(ref).max())
        assert np.abs(dual[b] - ref).max() <= bound
