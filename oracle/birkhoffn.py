"""fp64 CPU oracle for batched n x n Birkhoff projection (n = 2 .. 16).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` use it. The product path never imports it, and it
imports nothing from the product package or from the 4 x 4 oracle.

The arithmetic lives in ``birkhoffn_oracle.c`` (plain C, double precision, one
matrix at a time); this module marshals NumPy arrays and splits a batch across
threads.

  fwd(H, tol, max_iter) -> P, dual, iters   eq. birkhoff_projection via damped Newton on
                                            eq. min_fx with eq. grad_hess (a = b = 1, eta = 1)
  bwd(P, dP) -> dH                          eq. derivative (a = b = 1, eta = 1), sign of R = -M
  sinkhorn(H, tol, max_steps) -> P, steps   eq. sinkhorn_knopp run to a row-sum tolerance

General entropic OT (eq. entropic with cost M, marginals a, b, regulariser eta):
  ot_fwd(M, a, b, eta) -> T, dual, iters    the same damped Newton on eq. min_fx with the
                                            general eq. grad_hess; dual = (alpha, beta), beta_n = 0
  ot_bwd(T, a, G, eta) -> dM                eq. derivative (dL/dM)
  ot_sinkhorn(M, a, b, eta) -> T, steps     u = a / (K v), v = b / (K^T u), K = exp(-M / eta)
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "birkhoffn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle_birkhoffn.so")
_lib = None

DEFAULT_TOL = 1e-13
DEFAULT_MAX_ITER = 10000
NMAX = 16


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
        i32, i64 = ctypes.c_int, ctypes.c_int64
        lib.oraclen_fwd.argtypes = [i32, dp, dp, dp, ip, i64, i64, ctypes.c_double, i32]
        lib.oraclen_bwd.argtypes = [i32, dp, dp, dp, i64, i64]
        lib.oraclen_sinkhorn.argtypes = [i32, dp, dp, ip, i64, i64, ctypes.c_double, i32]
        d = ctypes.c_double
        lib.oraclen_ot_fwd.argtypes = [i32, dp, dp, dp, d, dp, dp, ip, i64, i64, d, i32]
        lib.oraclen_ot_bwd.argtypes = [i32, dp, dp, d, dp, dp, i64, i64]
        lib.oraclen_ot_sinkhorn.argtypes = [i32, dp, dp, dp, d, dp, ip, i64, i64, d, i32]
        for f in (lib.oraclen_fwd, lib.oraclen_bwd, lib.oraclen_sinkhorn, lib.oraclen_ot_fwd,
                  lib.oraclen_ot_bwd, lib.oraclen_ot_sinkhorn):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(x) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    if a.ndim != 3 or a.shape[1] != a.shape[2] or not 2 <= a.shape[1] <= NMAX:
        raise ValueError(f"expected [B, n, n] with 2 <= n <= {NMAX}, got {a.shape}")
    return a


def _ptr(a: np.ndarray, ty=ctypes.c_double):
    return a.ctypes.data_as(ctypes.POINTER(ty))


def _threads(threads):
    return max(1, min(16, os.cpu_count() or 1)) if threads is None else threads


def _ranges(B: int, threads: int):
    threads = max(1, min(threads, B // 64 if B >= 64 else 1))
    edges = np.linspace(0, B, threads + 1).astype(np.int64)
    return [(int(a), int(b)) for a, b in zip(edges[:-1], edges[1:]) if b > a]


def _run(fn, B, threads):
    if B:
        with ThreadPoolExecutor(_threads(threads)) as ex:
            list(ex.map(fn, _ranges(B, _threads(threads))))


def fwd(H, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER, threads: int | None = None):
    """Project exp(H[b]) onto the Birkhoff polytope, fp64.

    Returns (P [B,n,n], dual [B,2n] = (alpha_1..n, beta_1..n-1, 0),
    iters [B] int32: updates applied, -1 not converged, -2 non-finite input).
    """
    lib = _load()
    H = _f64(H)
    B, n = H.shape[0], H.shape[1]
    P = np.empty_like(H)
    dual = np.empty((B, 2 * n), np.float64)
    iters = np.empty(B, np.int32)
    _run(lambda r: lib.oraclen_fwd(n, _ptr(H), _ptr(P), _ptr(dual), _ptr(iters, ctypes.c_int32),
                                   r[0], r[1], tol, max_iter), B, threads)
    return P, dual, iters


def bwd(P, dP, threads: int | None = None) -> np.ndarray:
    """dH = (dP/dH)^T dP at the projection P (eq. derivative, sign flipped for R = -M)."""
    lib = _load()
    P = _f64(P)
    G = _f64(dP)
    if G.shape != P.shape:
        raise ValueError("P and dP differ in shape")
    B, n = P.shape[0], P.shape[1]
    dH = np.empty_like(P)
    _run(lambda r: lib.oraclen_bwd(n, _ptr(P), _ptr(G), _ptr(dH), r[0], r[1]), B, threads)
    return dH


def sinkhorn(H, tol: float = 1e-14, max_steps: int = 1_000_000, threads: int | None = None):
    """diag(u) exp(H) diag(v) from Sinkhorn-Knopp steps (v = 1 first) until the row
    sums are within tol of one; returns (P, steps)."""
    lib = _load()
    H = _f64(H)
    B, n = H.shape[0], H.shape[1]
    P = np.empty_like(H)
    steps = np.empty(B, np.int32)
    _run(lambda r: lib.oraclen_sinkhorn(n, _ptr(H), _ptr(P), _ptr(steps, ctypes.c_int32),
                                        r[0], r[1], tol, max_steps), B, threads)
    return P, steps


def marginal_errors(P) -> np.ndarray:
    """Per matrix: max over rows and columns of |sum - 1|, in fp64."""
    P = _f64(P)
    return np.maximum(np.abs(P.sum(axis=2) - 1.0).max(axis=1), np.abs(P.sum(axis=1) - 1.0).max(axis=1))


def _marg(x, B, n, name):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    if a.shape != (B, n):
        raise ValueError(f"{name} must have shape {(B, n)}, got {a.shape}")
    return a


def ot_fwd(M, a, b, eta: float = 1.0, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER,
           threads: int | None = None):
    """Entropic OT per matrix: T = argmin <T, M> - eta h(T) over Pi(a[b], b[b]), fp64.

    Returns (T [B,n,n], dual [B,2n] = (alpha_1..n, beta_1..n-1, 0), iters [B] int32)."""
    lib = _load()
    M = _f64(M)
    B, n = M.shape[0], M.shape[1]
    a = _marg(a, B, n, "a")
    b = _marg(b, B, n, "b")
    T = np.empty_like(M)
    dual = np.empty((B, 2 * n), np.float64)
    iters = np.empty(B, np.int32)
    rc = []
    _run(lambda r: rc.append(lib.oraclen_ot_fwd(n, _ptr(M), _ptr(a), _ptr(b), float(eta), _ptr(T), _ptr(dual),
                                                _ptr(iters, ctypes.c_int32), r[0], r[1], tol, max_iter)),
         B, threads)
    if any(rc):
        raise ValueError("eta must be positive")
    return T, dual, iters


def ot_bwd(T, a, G, eta: float = 1.0, threads: int | None = None) -> np.ndarray:
    """dL/dM at the OT solution T (eq. derivative) for upstream gradient G = dL/dT."""
    lib = _load()
    T = _f64(T)
    G = _f64(G)
    B, n = T.shape[0], T.shape[1]
    a = _marg(a, B, n, "a")
    dM = np.empty_like(T)
    _run(lambda r: lib.oraclen_ot_bwd(n, _ptr(T), _ptr(a), float(eta), _ptr(G), _ptr(dM), r[0], r[1]),
         B, threads)
    return dM


def ot_sinkhorn(M, a, b, eta: float = 1.0, tol: float = 1e-14, max_steps: int = 1_000_000,
                threads: int | None = None):
    """Sinkhorn iterations with marginals until the row sums are within tol of a."""
    lib = _load()
    M = _f64(M)
    B, n = M.shape[0], M.shape[1]
    a = _marg(a, B, n, "a")
    b = _marg(b, B, n, "b")
    T = np.empty_like(M)
    steps = np.empty(B, np.int32)
    _run(lambda r: lib.oraclen_ot_sinkhorn(n, _ptr(M), _ptr(a), _ptr(b), float(eta), _ptr(T),
                                           _ptr(steps, ctypes.c_int32), r[0], r[1], tol, max_steps),
         B, threads)
    return T, steps
