"""fp64 CPU oracle for the residual mixing of the mHC layer.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the CPU baseline
leg of ``bench.py`` use it. The product path never imports it, and it imports nothing
from the product package.

Sec. 2.1 writes the layer update as x_{l+1} = H^res x_l + (H^post)^T F(H^pre x_l), with
x_l the n x C matrix of a token's n streams, and (mHC) H^res the projection of
exp(H~^res) onto the Birkhoff polytope. The mixing term for one token is therefore the
matrix product Y = P X with P = proj(exp(H)) (eq. birkhoff_projection, computed by the
4x4 oracle) and X the token's 4 x C streams. Its gradients are those of a matrix product,
dX = P^T dY and dP = dY X^T, and dH is the projection's gradient (eq. derivative,
the 4x4 oracle's bwd) applied to that dP.

Functions (n streams per token: the 4 x 4 oracle for n = 4, the size-generic one otherwise):
  mix_fwd(H, X, tol) -> Y, P       Y[b] = P[b] @ X[b]
  mix_bwd(P, X, dY) -> dX, dH      dX[b] = P[b]^T @ dY[b], dH = bwd(P, dY @ X^T)
"""
from __future__ import annotations

import numpy as np

from . import birkhoffn, bwd, fwd


def _projection(n: int):
    """The 4 x 4 oracle for n = 4, the size-generic one otherwise."""
    return (fwd, bwd) if n == 4 else (birkhoffn.fwd, birkhoffn.bwd)


def mix_fwd(H: np.ndarray, X: np.ndarray, tol: float | None = None, threads: int | None = None):
    """H [B, n, n], X [B, n, C] (any float dtype; computed in fp64). Returns (Y, P)."""
    H = np.asarray(H, dtype=np.float64)
    kw = {} if tol is None else {"tol": tol}
    if threads is not None:
        kw["threads"] = threads
    P, _, _ = _projection(H.shape[-1])[0](H, **kw)
    Y = np.matmul(P, np.asarray(X, dtype=np.float64))
    return Y, P


def mix_bwd(P: np.ndarray, X: np.ndarray, dY: np.ndarray, threads: int | None = None):
    """From the forward's P [B, n, n], X and dY [B, n, C]: (dX [B, n, C], dH [B, n, n])."""
    P = np.asarray(P, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    dX = np.matmul(np.swapaxes(P, -1, -2), dY)
    dP = np.matmul(dY, np.swapaxes(X, -1, -2))
    kw = {} if threads is None else {"threads": threads}
    return dX, _projection(P.shape[-1])[1](P, dP, **kw)
