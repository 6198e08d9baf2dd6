"""The per-matrix dual bound used by the GPU parity tests, checked on the CPU.

A solution stopped at column residual 1e-6 (the oracle itself at tol 1e-6) must fall within
the bound of the exact dual (the oracle at 1e-13); the bound must be tight enough to decide
something (well-conditioned matrices are determined), and a dual moved by a small constant on
one potential must fail it where the dual is determined.
"""
import numpy as np
import pytest

import oracle
import workloads
from tests._gpu import dual_bound


@pytest.mark.parametrize("sigma", [0.1, 1.0, 5.0, 20.0, 50.0])
def test_tol_solution_within_bound(sigma):
    H, _ = workloads.gauss(2000, sigma, seed=11)
    H = H.astype(np.float64)
    Pr, dr, _ = oracle.fwd(H)
    Pl, dl, it = oracle.fwd(H, tol=1e-6)
    assert (it >= 0).all()
    b = dual_bound(Pr, dr)
    assert (np.abs(dl - dr).max(axis=1) <= b).all()


def test_bound_decides_and_detects():
    H, _ = workloads.gauss(2000, 1.0, seed=12)
    H = H.astype(np.float64)
    Pr, dr, _ = oracle.fwd(H)
    b = dual_bound(Pr, dr)
    assert (b <= 1e-3).mean() > 0.99          # N(0,1) logits: the dual is determined
    bad = dr.copy()
    bad[:, 5] += 2e-3                          # beta_2 off by 2e-3 (alpha left as it was)
    assert (np.abs(bad - dr).max(axis=1) > b).mean() > 0.99


def test_weakly_coupled_columns_are_not_gated():
    # near permutations: the column graph's weights are ~e^-40, the dual is not determined in fp32
    H, _ = workloads.near_permutation(500, 20.0, 0.1, seed=13)
    Pr, dr, _ = oracle.fwd(H.astype(np.float64))
    assert (dual_bound(Pr, dr) > 1.0).all()
