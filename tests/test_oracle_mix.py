"""Pins for the residual-mixing oracle (CPU only).

The mixing term of the mHC update (Sec. 2.1) is Y = P X per token, P doubly stochastic. The
pins check it against what the Birkhoff constraint fixes (identical streams pass through,
the streams' total is conserved, separable logits average the streams, near-permutation
logits permute them), against plain loops on tiny inputs, against central finite
differences of the whole map (H, X) -> Y, and against the adjoint identity that separates
dX = P^T dY from P dY.
"""
import numpy as np
import pytest

import oracle
from oracle.mix import mix_bwd, mix_fwd
import workloads


def _streams(B, C, seed):
    return np.random.default_rng(seed).standard_normal((B, 4, C))


@pytest.mark.parametrize("sigma", [1.0, 10.0])
def test_identical_streams_pass_through(sigma):
    # rows of P sum to one: if every stream equals v, every output stream equals v
    H, _ = workloads.gauss(50, sigma, seed=1)
    v = np.random.default_rng(2).standard_normal((50, 1, 7))
    Y, _ = mix_fwd(H, np.repeat(v, 4, axis=1))
    assert np.abs(Y - v).max() < 1e-11


@pytest.mark.parametrize("sigma", [1.0, 10.0])
def test_total_of_streams_conserved(sigma):
    # columns of P sum to one: sum_i Y_i = sum_j X_j
    H, _ = workloads.gauss(50, sigma, seed=3)
    X = _streams(50, 9, 4)
    Y, _ = mix_fwd(H, X)
    assert np.abs(Y.sum(axis=1) - X.sum(axis=1)).max() < 1e-11


def test_separable_logits_average_the_streams():
    rng = np.random.default_rng(5)
    H = rng.standard_normal((20, 4, 1)) + rng.standard_normal((20, 1, 4))
    X = _streams(20, 6, 6)
    Y, _ = mix_fwd(H, X)
    assert np.abs(Y - X.mean(axis=1, keepdims=True)).max() < 1e-12


def test_near_permutation_logits_permute_the_streams():
    rng = np.random.default_rng(7)
    perms = np.stack([rng.permutation(4) for _ in range(30)])
    H = np.zeros((30, 4, 4))
    H[np.arange(30)[:, None], np.arange(4)[None, :], perms] = 30.0
    X = _streams(30, 5, 8)
    Y, _ = mix_fwd(H, X)
    # Y_i = X_{perm(i)} up to the e^-30 off-permutation mass
    assert np.abs(Y - X[np.arange(30)[:, None], perms]).max() < 1e-11


def test_against_loops():
    H, _ = workloads.gauss(3, 3.0, seed=9)
    X = _streams(3, 5, 10)
    G = _streams(3, 5, 11)
    Y, P = mix_fwd(H, X)
    dX, dH = mix_bwd(P, X, G)
    for b in range(3):
        for i in range(4):
            for c in range(5):
                assert abs(Y[b, i, c] - sum(P[b, i, j] * X[b, j, c] for j in range(4))) < 1e-14
                assert abs(dX[b, i, c] - sum(P[b, j, i] * G[b, j, c] for j in range(4))) < 1e-14
    dP = np.zeros((3, 4, 4))
    for b in range(3):
        for i in range(4):
            for j in range(4):
                dP[b, i, j] = sum(G[b, i, c] * X[b, j, c] for c in range(5))
    assert np.abs(dH - oracle.bwd(P, dP)).max() < 1e-14


def test_adjoint_identity():
    # <dY, P X> = <P^T dY, X> for every X: fails for dX = P dY unless P is symmetric
    H, _ = workloads.gauss(40, 5.0, seed=12)
    X = _streams(40, 8, 13)
    G = _streams(40, 8, 14)
    Y, P = mix_fwd(H, X)
    dX, _ = mix_bwd(P, X, G)
    lhs = (G * Y).sum(axis=(1, 2))
    rhs = (dX * X).sum(axis=(1, 2))
    assert np.abs(lhs - rhs).max() < 1e-12
    assert np.abs(P - np.swapaxes(P, 1, 2)).max() > 1e-2  # the inputs do tell P from P^T


@pytest.mark.parametrize("sigma", [0.5, 3.0, 10.0])
def test_finite_differences(sigma):
    # L(H, X) = <G, Y(H, X)>: central differences in every entry of H and of X
    B, C = 6, 3
    H, _ = workloads.gauss(B, sigma, seed=15)
    H = H.astype(np.float64)
    X = _streams(B, C, 16)
    G = _streams(B, C, 17)
    _, P = mix_fwd(H, X, tol=1e-14)
    dX, dH = mix_bwd(P, X, G)
    h = 1e-5

    def loss(Hh, Xx):
        Y, _ = mix_fwd(Hh, Xx, tol=1e-14)
        return (G * Y).sum(axis=(1, 2))
    fdH = np.zeros_like(H)
    for k in range(16):
        E = np.zeros((4, 4))
        E[divmod(k, 4)] = h
        fdH[:, k // 4, k % 4] = (loss(H + E, X) - loss(H - E, X)) / (2 * h)
    fdX = np.zeros_like(X)
    for k in range(4 * C):
        E = np.zeros((4, C))
        E[divmod(k, C)] = h
        fdX[:, k // C, k % C] = (loss(H, X + E) - loss(H, X - E)) / (2 * h)
    scale = np.maximum(1.0, np.abs(fdH).max(axis=(1, 2)))
    assert (np.abs(dH - fdH).max(axis=(1, 2)) / scale).max() < 1e-7
    assert np.abs(dX - fdX).max() < 1e-8


# n = 8 streams (the size-generic projection oracle)
def _logits8(B, sigma, seed):
    return sigma * np.random.default_rng(seed).standard_normal((B, 8, 8))


def test_n8_structure():
    H = _logits8(40, 5.0, 20)
    rng = np.random.default_rng(21)
    v = rng.standard_normal((40, 1, 6))
    Y, _ = mix_fwd(H, np.repeat(v, 8, axis=1))
    assert np.abs(Y - v).max() < 1e-11                       # unit row sums
    X = rng.standard_normal((40, 8, 6))
    Y, P = mix_fwd(H, X)
    assert np.abs(Y.sum(axis=1) - X.sum(axis=1)).max() < 1e-11  # unit column sums
    Hs = rng.standard_normal((10, 8, 1)) + rng.standard_normal((10, 1, 8))
    Ys, _ = mix_fwd(Hs, X[:10])
    assert np.abs(Ys - X[:10].mean(axis=1, keepdims=True)).max() < 1e-12
    G = rng.standard_normal((40, 8, 6))
    dX, _ = mix_bwd(P, X, G)
    assert np.abs((G * Y).sum(axis=(1, 2)) - (dX * X).sum(axis=(1, 2))).max() < 1e-12


def test_n8_finite_differences():
    B, C = 3, 2
    H = _logits8(B, 2.0, 22)
    rng = np.random.default_rng(23)
    X = rng.standard_normal((B, 8, C))
    G = rng.standard_normal((B, 8, C))
    _, P = mix_fwd(H, X, tol=1e-14)
    dX, dH = mix_bwd(P, X, G)
    h = 1e-5

    def loss(Hh, Xx):
        Y, _ = mix_fwd(Hh, Xx, tol=1e-14)
        return (G * Y).sum(axis=(1, 2))
    fdH = np.zeros_like(H)
    for k in range(64):
        E = np.zeros((8, 8))
        E[divmod(k, 8)] = h
        fdH[:, k // 8, k % 8] = (loss(H + E, X) - loss(H - E, X)) / (2 * h)
    fdX = np.zeros_like(X)
    for k in range(8 * C):
        E = np.zeros((8, C))
        E[divmod(k, C)] = h
        fdX[:, k // C, k % C] = (loss(H, X + E) - loss(H, X - E)) / (2 * h)
    scale = np.maximum(1.0, np.abs(fdH).max(axis=(1, 2)))
    assert (np.abs(dH - fdH).max(axis=(1, 2)) / scale).max() < 1e-7
    assert np.abs(dX - fdX).max() < 1e-8
