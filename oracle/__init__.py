"""fp64 CPU oracle for the batched 4x4 Birkhoff projection.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` use it. The product path never imports it, and it
imports nothing from the product package.

The arithmetic lives in ``birkhoff4_oracle.c`` (plain C, double precision, one
matrix at a time); this module only marshals NumPy arrays and splits a batch
across threads (ctypes releases the GIL during foreign calls).

Functions (paper references are to sections/equations):
  fwd(H, tol, max_iter) -> P, dual, iters   KL projection, eq. birkhoff_projection,
                                            via damped Newton on eq. min_fx
  bwd(P, dP) -> dH                          implicit-differentiation vJP, eq. derivative
  sk_fwd(H, n) / sk_bwd(H, dP, n)           n-step Sinkhorn-Knopp, eq. sinkhorn_knopp,
                                            and the gradient of that n-step map
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "birkhoff4_oracle.c")
_LIB = os.path.join(_HERE, "liboracle_birkhoff4.so")
_lib = None

DEFAULT_TOL = 1e-13
DEFAULT_MAX_ITER = 10000


def build(force: bool = False) -> str:
    """Compile the oracle with the host C compiler (plain -O2, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math",
             "-ffp-contract=off", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        lib.oracle_fwd.argtypes = [dp, dp, dp, ip, ctypes.c_int64, ctypes.c_double, ctypes.c_int]
        lib.oracle_fwd.restype = ctypes.c_int
        lib.oracle_bwd.argtypes = [dp, dp, dp, ctypes.c_int64]
        lib.oracle_bwd.restype = None
        lib.oracle_sk_fwd.argtypes = [dp, dp, ctypes.c_int64, ctypes.c_int]
        lib.oracle_sk_fwd.restype = ctypes.c_int
        lib.oracle_sk_bwd.argtypes = [dp, dp, dp, ctypes.c_int64, ctypes.c_int]
        lib.oracle_sk_bwd.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(x) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64)).reshape(-1, 4, 4)
    return a


def _ptr(a: np.ndarray, ty=ctypes.c_double):
    return a.ctypes.data_as(ctypes.POINTER(ty))


def _split(B: int, threads: int):
    threads = max(1, min(threads, B // 256 if B >= 256 else 1))
    edges = np.linspace(0, B, threads + 1).astype(np.int64)
    return [(int(a), int(b)) for a, b in zip(edges[:-1], edges[1:]) if b > a]


def default_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def fwd(H, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER, threads: int | None = None):
    """Project exp(H[b]) onto the Birkhoff polytope in fp64.

    Returns (P [B,4,4] f64, dual [B,8] f64 = (alpha_1..4, beta_1..3, 0),
    iters [B] int32: updates applied, -1 not converged, -2 non-finite input).
    """
    lib = _load()
    H = _f64(H)
    B = H.shape[0]
    P = np.empty_like(H)
    dual = np.empty((B, 8), np.float64)
    iters = np.empty(B, np.int32)
    threads = default_threads() if threads is None else threads

    def run(r):
        a, b = r
        lib.oracle_fwd(_ptr(H[a:b]), _ptr(P[a:b]), _ptr(dual[a:b]),
                       _ptr(iters[a:b], ctypes.c_int32), b - a, tol, max_iter)

    if B:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, _split(B, threads)))
    return P, dual, iters


def bwd(P, dP, threads: int | None = None):
    """dH = (dP/dH)^T dP at the projection P (eq. derivative, sign flipped for R = -M)."""
    lib = _load()
    P = _f64(P)
    G = _f64(dP)
    B = P.shape[0]
    dH = np.empty_like(P)
    threads = default_threads() if threads is None else threads

    def run(r):
        a, b = r
        lib.oracle_bwd(_ptr(P[a:b]), _ptr(G[a:b]), _ptr(dH[a:b]), b - a)

    if B:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, _split(B, threads)))
    return dH


def sk_fwd(H, n_steps: int = 20) -> np.ndarray:
    """diag(u) exp(H) diag(v) after n_steps Sinkhorn-Knopp steps from v = 1."""
    lib = _load()
    H = _f64(H)
    P = np.empty_like(H)
    if lib.oracle_sk_fwd(_ptr(H), _ptr(P), H.shape[0], n_steps) != 0:
        raise ValueError("n_steps out of range")
    return P


def sk_bwd(H, dP, n_steps: int = 20) -> np.ndarray:
    """Exact gradient of the n_steps Sinkhorn-Knopp map, applied to dP."""
    lib = _load()
    H = _f64(H)
    G = _f64(dP)
    dH = np.empty_like(H)
    if lib.oracle_sk_bwd(_ptr(H), _ptr(G), _ptr(dH), H.shape[0], n_steps) != 0:
        raise ValueError("n_steps out of range")
    return dH


def marginal_errors(P) -> tuple[np.ndarray, np.ndarray]:
    """Per matrix: (max_i |r_i - 1| v max_j |c_j - 1|, Err = ||r-1||_1 + ||c-1||_1), in fp64.

    Err is the paper's marginal error (Sec. 5); the first value is its L-inf analogue.
    """
    P = _f64(P)
    r = P.sum(axis=2) - 1.0
    c = P.sum(axis=1) - 1.0
    linf = np.maximum(np.abs(r).max(axis=1), np.abs(c).max(axis=1))
    l1 = np.abs(r).sum(axis=1) + np.abs(c).sum(axis=1)
    return linf, l1
