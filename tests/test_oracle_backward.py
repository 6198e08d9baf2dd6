"""Pins for the oracle's implicit-differentiation backward (CPU only).

The oracle evaluates eq. derivative in rearranged, cancellation-free forms. These
tests pin it against independent routes: central finite differences of the
forward projection, the KKT-linearisation Jacobian, the closed form at
separable H, structural identities of the vector-Jacobian product, and the
paper's literal formula evaluated in high-precision decimals.
"""
import numpy as np
import pytest

import oracle
import workloads
from tests import _refs


def _proj(H, tol=1e-14):
    P, _, it = oracle.fwd(H, tol=tol)
    assert (it >= 0).all()
    return P


@pytest.mark.parametrize("sigma", [0.1, 1.0, 5.0, 20.0])
def test_finite_differences(sigma):
    H, G = workloads.gauss(32, sigma, seed=21)
    H = H.astype(np.float64)
    G = G.astype(np.float64)
    P = _proj(H)
    dH = oracle.bwd(P, G)
    h = 1e-5
    fd = np.zeros_like(H)
    for kl in range(16):
        k, l = divmod(kl, 4)
        E = np.zeros((4, 4))
        E[k, l] = h
        dPdh = (_proj(H + E) - _proj(H - E)) / (2 * h)
        fd[:, k, l] = (G * dPdh).sum(axis=(1, 2))
    scale = np.maximum(1.0, np.abs(fd).max(axis=(1, 2)))
    assert (np.abs(dH - fd).max(axis=(1, 2)) / scale).max() < 2e-7


@pytest.mark.parametrize("sigma", [0.5, 3.0, 8.0])
def test_kkt_linearisation_jacobian(sigma):
    H, G = workloads.gauss(200, sigma, seed=22)
    P = _proj(H.astype(np.float64))
    J = _refs.kkt_jacobian(P)
    vjp = np.einsum("bij,bi->bj", J, G.reshape(-1, 16).astype(np.float64)).reshape(-1, 4, 4)
    dH = oracle.bwd(P, G)
    assert np.abs(dH - vjp).max() < 1e-10


def test_separable_closed_form():
    # At T = J/4: dH = 1/4 (I - J/4) G (I - J/4)
    rng = np.random.default_rng(23)
    a = 5 * rng.standard_normal((50, 4, 1))
    b = 5 * rng.standard_normal((50, 1, 4))
    G = rng.standard_normal((50, 4, 4))
    P = _proj(a + b)
    C = np.eye(4) - 0.25
    expect = 0.25 * C @ G @ C
    assert np.abs(oracle.bwd(P, G) - expect).max() < 1e-13


@pytest.mark.parametrize("sigma", [1.0, 10.0, 50.0])
def test_vjp_structure(sigma):
    """Zero row/column sums; invariance to G + a1^T + 1b^T; symmetric PSD map.

    P(H) is the gradient of the convex function max_P <P,H> + h(P) (entropy h,
    Sec. 2.3), so dP/dH is symmetric positive semidefinite, and P is unchanged
    by additive row/column shifts of H.
    """
    H, G1 = workloads.gauss(500, sigma, seed=24)
    _, G2 = workloads.gauss(500, sigma, seed=25)
    H, G1, G2 = (x.astype(np.float64) for x in (H, G1, G2))
    P = _proj(H, tol=1e-13)
    d1 = oracle.bwd(P, G1)
    d2 = oracle.bwd(P, G2)
    scale = max(1.0, np.abs(d1).max())
    assert np.abs(d1.sum(axis=1)).max() < 1e-12 * scale
    assert np.abs(d1.sum(axis=2)).max() < 1e-12 * scale
    rng = np.random.default_rng(26)
    Gs = G1 + rng.standard_normal((500, 4, 1)) + rng.standard_normal((500, 1, 4))
    assert np.abs(oracle.bwd(P, Gs) - d1).max() < 1e-12 * scale
    s12 = (G1 * d2).sum(axis=(1, 2))
    s21 = (G2 * d1).sum(axis=(1, 2))
    assert np.abs(s12 - s21).max() < 1e-12
    assert ((G1 * d1).sum(axis=(1, 2)) >= -1e-14).all()


def test_permutation_equivariance():
    rng = np.random.default_rng(27)
    H = 8 * rng.standard_normal((300, 4, 4))
    G = rng.standard_normal((300, 4, 4))
    P = _proj(H)
    d = oracle.bwd(P, G)
    pr, pc = rng.permutation(4), rng.permutation(4)
    Pp = _proj(H[:, pr][:, :, pc])
    dp = oracle.bwd(Pp, G[:, pr][:, :, pc])
    assert np.abs(dp - d[:, pr][:, :, pc]).max() < 1e-10


@pytest.mark.parametrize("sigma,prec", [(5.0, 60), (20.0, 80), (50.0, 120)])
def test_literal_formula_high_precision(sigma, prec):
    """eq. derivative written literally (diag(b) - T^T T, Cramer's rule, D), in
    decimals at the polished T*, against the oracle's fp64 rearrangement."""
    H, G = workloads.gauss(6, sigma, seed=28)
    H = H.astype(np.float64)
    P, dual, _ = oracle.fwd(H)
    dH = oracle.bwd(P, G)
    for b in range(H.shape[0]):
        T = _refs.literal_newton_decimal(H[b], beta0=dual[b, 4:], prec=prec, tol_exp=prec // 2)
        ref = _refs.literal_backward_decimal(T, G[b], prec=prec)
        assert np.abs(dH[b] - ref).max() < 1e-11


def test_near_permutation_bounded():
    """Close to a permutation the vJP is tiny and bounded (dH_ij carries a factor
    T_ij times an O(|G|) term); rounding must not blow it up."""
    H, G = workloads.near_permutation(5000, 40.0, 0.1, seed=29)
    P = _proj(H.astype(np.float64), tol=1e-13)
    dH = oracle.bwd(P, G)
    assert np.isfinite(dH).all()
    assert np.abs(dH).max() < 1e-12
    ch = workloads.make_chunk(workloads.WORKLOADS["logunif_b2e25"], 0, B=200000)
    P, _, _ = oracle.fwd(ch.H)
    dH = oracle.bwd(P, ch.dP)
    assert np.abs(dH).max() < 3 * np.abs(ch.dP).max()


@pytest.mark.parametrize("family,scale", [("gauss", 0.3), ("gauss", 1.0), ("gauss", 20.0), ("uniform", 1.0),
                                          ("uniform", 10.0)])
def test_literal_formula_from_independent_start(family, scale):
    """eq. derivative written literally, at a T* that the literal Newton reached from
    beta = 0 (independent of the oracle's forward), against the oracle's backward."""
    prec = 60 if scale <= 5 else 80
    gen = workloads.gauss if family == "gauss" else workloads.uniform
    H, G = gen(8, scale, seed=31)
    H = H.astype(np.float64)
    P, _, _ = oracle.fwd(H)
    dH = oracle.bwd(P, G)
    for b in range(H.shape[0]):
        T = _refs.literal_newton_decimal(H[b], prec=prec, tol_exp=prec // 2)
        ref = _refs.literal_backward_decimal(T, G[b], prec=prec)
        assert np.abs(dH[b] - ref).max() < 1e-11
