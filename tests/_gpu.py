"""Helpers for the GPU parity tests: run the HIP path, run the oracle on the same
inputs, compare to the stated tolerances."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import paper_2606_07574_amd as b4

TOL_P = 1e-5        # max |P - P_ref|
TOL_DH = 1e-4       # per matrix: |dH - dH_ref|_inf / max(1, |dH_ref|_inf)
TOL_MARGINAL = 1e-5  # max row/column marginal error
MAX_ITER = 64
GPU_TOL = 1e-6      # the GPU's stopping tolerance in these tests
# Row and column sums of dH vanish in exact arithmetic; in fp32 they are bounded by the
# stopping tolerance times the size of the flows, so the check is relative to max|dH|.
TOL_DH_SUMS = 2e-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(x: np.ndarray, dtype=torch.float32) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x)).to(device="cuda:0", dtype=dtype)


def bits_to_dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda:0").view(torch.bfloat16)


VARIANTS = [b4.THROUGHPUT, b4.LATENCY]
VARIANT_IDS = ["throughput", "latency"]


def gpu_fwd(Hd: torch.Tensor, tol=GPU_TOL, max_iter=MAX_ITER, variant=b4.AUTO):
    P, dual, it = b4.fwd(Hd, tol, max_iter, want_dual=True, want_iters=True, variant=variant)
    torch.cuda.synchronize()
    return P, dual, it


def marginal_linf_device(P: torch.Tensor) -> torch.Tensor:
    """Per-matrix max(|row sum - 1|, |col sum - 1|), accumulated in fp64 on the device."""
    P64 = P.double()
    r = (P64.sum(dim=-1) - 1).abs().amax(dim=-1)
    c = (P64.sum(dim=-2) - 1).abs().amax(dim=-1)
    return torch.maximum(r, c)


def dh_sums_rel_device(dH: torch.Tensor) -> torch.Tensor:
    """Per matrix: max |row or column sum of dH| / max(1, max|dH|), in fp64 on the device."""
    d64 = dH.double()
    s = torch.maximum(d64.sum(dim=-1).abs().amax(dim=-1), d64.sum(dim=-2).abs().amax(dim=-1))
    return s / torch.clamp(d64.abs().amax(dim=(-2, -1)), min=1.0)


def dh_rel_err(dH: np.ndarray, ref: np.ndarray) -> np.ndarray:
    dH = dH.reshape(-1, 16)
    ref = ref.reshape(-1, 16)
    return np.abs(dH - ref).max(axis=1) / np.maximum(1.0, np.abs(ref).max(axis=1))


def dual_bound(Pr: np.ndarray, dualr: np.ndarray, tol: float = GPU_TOL) -> np.ndarray:
    """Per-matrix bound on |dual - dual_ref| for a solution that stopped at column residual tol.

    The reduced dual's Hessian at the solution is the Laplacian of the column graph with
    weights W_jk = sum_i P_ij P_ik, grounded at column 4 (eq. grad_hess with unit rows). A
    point whose column sums are off by delta c has potentials off by L^{-1} delta c to first
    order, and alpha_i = alpha*(beta) moves by sum_j P_ij delta beta_j, i.e. by at most
    |delta beta|_inf. The fp32 column sums of the stored P carry up to ~4e-6 of rounding on top
    of tol (product-form updates), and the fp32 accumulation of the potentials adds ~1e-6 of
    their size; both get a factor 2 of margin. Where L is near singular (weakly coupled
    columns) the dual is not determined in fp32 and the bound is vacuous."""
    W = np.einsum("bij,bik->bjk", Pr, Pr)
    W[:, np.arange(4), np.arange(4)] = 0.0
    deg = W.sum(axis=2)
    L = -W[:, :3, :3]
    L[:, np.arange(3), np.arange(3)] = deg[:, :3]
    with np.errstate(all="ignore"):
        sing = ~(np.abs(np.linalg.det(L)) > 0.0)  # exactly singular: every weight of a column underflowed
        L[sing] = np.eye(3)
        norm = np.abs(np.linalg.inv(L)).sum(axis=2).max(axis=1)
    norm = np.where(np.isfinite(norm) & ~sing, norm, np.inf)
    return 2.0 * norm * (tol + 4e-6) + 1e-5 * (1.0 + np.abs(dualr).max(axis=1))


def parity_arrays(H32: np.ndarray, Pg: np.ndarray, dualg: np.ndarray | None = None,
                  dP32: np.ndarray | None = None, dHg: np.ndarray | None = None) -> dict:
    """Per-matrix comparison of GPU outputs with the oracle on the same (fp32) inputs."""
    Pr, dualr, itr = oracle.fwd(H32.astype(np.float64))
    out = {"oracle_iters": itr,
           "p_err": np.abs(Pg.astype(np.float64) - Pr).reshape(-1, 16).max(axis=1)}
    out["marg"] = oracle.marginal_errors(Pg)[0]
    if dualg is not None:
        d64 = dualg.astype(np.float64)
        out["dual_err"] = np.abs(d64 - dualr).max(axis=1)
        out["dual_bound"] = dual_bound(Pr, dualr)
        out["beta4"] = d64[:, 7]
        # the reported dual reproduces P: log P - H = alpha_i + beta_j where P carries mass
        Pg64 = Pg.astype(np.float64)
        mask = Pg64 > 1e-4
        kkt = np.log(np.where(mask, Pg64, 1.0)) - H32 - d64[:, :4, None] - d64[:, None, 4:]
        scale = 1.0 + np.abs(H32).max(axis=(1, 2), keepdims=True)
        out["kkt"] = np.where(mask, np.abs(kkt) / scale, 0.0).reshape(-1, 16).max(axis=1)
    if dP32 is not None:
        ref = oracle.bwd(Pr, dP32.astype(np.float64))
        out["dh_err"] = dh_rel_err(dHg.astype(np.float64), ref)
    return out


def check_parity(H32: np.ndarray, Pg: np.ndarray, dualg: np.ndarray | None = None,
                 dP32: np.ndarray | None = None, dHg: np.ndarray | None = None, label: str = ""):
    """Compare GPU outputs with the oracle on the same (fp32-representable) inputs."""
    a = parity_arrays(H32, Pg, dualg, dP32, dHg)
    assert (a["oracle_iters"] >= 0).all(), f"{label}: oracle failed to converge"
    say(f"  [{label}] max|P-Pref|={a['p_err'].max():.3e} max marginal={a['marg'].max():.3e}")
    assert a["p_err"].max() <= TOL_P, f"{label}: max|P - P_ref| = {a['p_err'].max()}"
    assert a["marg"].max() <= TOL_MARGINAL, f"{label}: marginal {a['marg'].max()}"
    if dualg is not None:
        ratio = a["dual_err"] / a["dual_bound"]
        det = a["dual_bound"] <= 1e-3
        say(f"  [{label}] dual: max err/bound={ratio.max():.3f}, {det.sum()} of {len(det)} determined "
            f"(bound <= 1e-3), max err there={a['dual_err'][det].max() if det.any() else 0:.3e}; "
            f"kkt rel err={a['kkt'].max():.3e}")
        assert ratio.max() <= 1.0, f"{label}: dual differs from the oracle's beyond its bound"
        assert a["kkt"].max() < 2e-4
        assert (a["beta4"] == 0).all()
    if dP32 is not None:
        say(f"  [{label}] max dH rel err={a['dh_err'].max():.3e}")
        assert a["dh_err"].max() <= TOL_DH, f"{label}: dH rel err {a['dh_err'].max()}"
