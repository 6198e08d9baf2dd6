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


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(x: np.ndarray, dtype=torch.float32) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x)).to(device="cuda:0", dtype=dtype)


def bits_to_dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda:0").view(torch.bfloat16)


VARIANTS = [b4.THROUGHPUT, b4.LATENCY]
VARIANT_IDS = ["throughput", "latency"]


def gpu_fwd(Hd: torch.Tensor, tol=1e-6, max_iter=MAX_ITER, variant=b4.AUTO):
    P, dual, it = b4.fwd(Hd, tol, max_iter, want_dual=True, want_iters=True, variant=variant)
    torch.cuda.synchronize()
    return P, dual, it


def marginal_linf_device(P: torch.Tensor) -> torch.Tensor:
    """Per-matrix max(|row sum - 1|, |col sum - 1|), accumulated in fp64 on the device."""
    P64 = P.double()
    r = (P64.sum(dim=-1) - 1).abs().amax(dim=-1)
    c = (P64.sum(dim=-2) - 1).abs().amax(dim=-1)
    return torch.maximum(r, c)


def dh_rel_err(dH: np.ndarray, ref: np.ndarray) -> np.ndarray:
    dH = dH.reshape(-1, 16)
    ref = ref.reshape(-1, 16)
    return np.abs(dH - ref).max(axis=1) / np.maximum(1.0, np.abs(ref).max(axis=1))


def check_parity(H32: np.ndarray, Pg: np.ndarray, dualg: np.ndarray | None = None,
                 dP32: np.ndarray | None = None, dHg: np.ndarray | None = None, label: str = ""):
    """Compare GPU outputs with the oracle on the same (fp32-representable) inputs."""
    Pr, dualr, itr = oracle.fwd(H32.astype(np.float64))
    assert (itr >= 0).all(), f"{label}: oracle failed to converge"
    perr = np.abs(Pg.astype(np.float64) - Pr).max()
    linf, _ = oracle.marginal_errors(Pg)
    say(f"  [{label}] max|P-Pref|={perr:.3e} max marginal={linf.max():.3e}")
    assert perr <= TOL_P, f"{label}: max|P - P_ref| = {perr}"
    assert linf.max() <= TOL_MARGINAL, f"{label}: marginal {linf.max()}"
    if dualg is not None:
        # the reported dual reproduces P: log P - H = alpha_i + beta_j where P carries mass
        Pg64 = Pg.astype(np.float64)
        mask = Pg64 > 1e-4
        kkt = np.log(np.where(mask, Pg64, 1.0)) - H32 - dualg[:, :4, None] - dualg[:, None, 4:]
        scale = 1.0 + np.abs(H32).max(axis=(1, 2), keepdims=True)
        kerr = (np.abs(kkt) / scale)[mask].max()
        say(f"  [{label}] dual kkt rel err={kerr:.3e}")
        assert kerr < 2e-4
        assert (dualg[:, 7] == 0).all()
    if dP32 is not None:
        ref = oracle.bwd(Pr, dP32.astype(np.float64))
        e = dh_rel_err(dHg.astype(np.float64), ref)
        say(f"  [{label}] max dH rel err={e.max():.3e}")
        assert e.max() <= TOL_DH, f"{label}: dH rel err {e.max()}"
