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

Functions:
  mix_fwd(H, X, tol) -> Y, P       Y[b] = P[b] @ X[b]
  mix_bwd(P, X, dY) -> dX, dH      dX[b] = P[b]^T @ dY[b], dH = bwd(P, dY @ X^T)
"""
from __future__ import annotations

import numpy as np

from . import bwd, fwd


def mix_fwd(H: np.ndarray, X: np.ndarray, tol: float | None = None, threads: int | None = None):
    """H [B, 4, 4], X [B, 4, C] (any float dtype; computed in fp64). Returns (Y, P)."""
    kw = {} if tol is None else {"tol": tol}
    if threads is not None:
        kw["threads"] = threads
    P, _, _ = fwd(np.asarray(H, dtype=np.float64), **kw)
    Y = np.matmul(P, np.asarray(X, dtype=np.float64))
    return Y, P


def mix_bwd(P: np.ndarray, X: np.ndarray, dY: np.ndarray, threads: int | None = None):
    """From the forward's P [B, 4, 4], X and dY [B, 4, C]: (dX [B, 4, C], dH [B, 4, 4])."""
    P = np.asarray(P, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    dX = np.matmul(np.swapaxes(P, -1, -2), dY)
    dP = np.matmul(dY, np.swapaxes(X, -1, -2))
    kw = {} if threads is None else {"threads": threads}
    return dX, bwd(P, dP, **kw)
