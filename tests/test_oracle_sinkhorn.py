"""Pins for the oracle's n-step Sinkhorn-Knopp baseline (CPU only).

* golden: the paper's Table 2 marginal-error statistics of 20-step SK on
  N(0,10^2) and Unif(-10,10) inputs (large magnitudes, where the error is set by
  the iteration's convergence rather than by rounding);
* the n -> infinity limit is the Birkhoff projection (eq. bca converges);
* exact structure: unit column sums after every full step, invariance to row
  shifts of H;
* the gradient of the n-step map: central finite differences, and torch
  autograd (float64, CPU) through a plain n-step loop.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "sk20_table2.json")


@pytest.mark.parametrize("row,draw", [
    ("normal_sd10", lambda r, n: 10.0 * r.standard_normal((n, 4, 4))),
    ("uniform_pm10", lambda r, n: r.uniform(-10.0, 10.0, (n, 4, 4))),
])
def test_table2_statistics(row, draw):
    ref = json.load(open(GOLDEN))
    scale = ref["scale"]
    paper = ref["rows"][row]["vanilla"]
    rng = np.random.default_rng(np.random.SeedSequence([0, 31, len(row)]))
    H = draw(rng, 10000)
    _, err = oracle.marginal_errors(oracle.sk_fwd(H, 20))
    assert abs(err.mean() / (paper["mean"] * scale) - 1) < 0.05
    assert abs(np.median(err) / (paper["median"] * scale) - 1) < 0.05
    assert abs(err.std() / (paper["std"] * scale) - 1) < 0.10


def test_limit_is_projection():
    H, _ = workloads.gauss(200, 1.0, seed=32)
    P = oracle.sk_fwd(H, 200)
    Pn, _, _ = oracle.fwd(H)
    assert np.abs(P - Pn).max() < 1e-12


def test_structure():
    H, _ = workloads.gauss(300, 5.0, seed=33)
    H = H.astype(np.float64)
    for n in [1, 2, 20]:
        P = oracle.sk_fwd(H, n)
        assert np.abs(P.sum(axis=1) - 1).max() < 1e-14
        shift = np.random.default_rng(n).standard_normal((300, 4, 1)) * 30
        assert np.abs(oracle.sk_fwd(H + shift, n) - P).max() < 1e-13
    # zero steps: A = exp(H) row-scaled by its maxima (no normalisation yet)
    P0 = oracle.sk_fwd(H, 0)
    assert np.abs(P0 - np.exp(H - H.max(axis=2, keepdims=True))).max() < 1e-15


@pytest.mark.parametrize("sigma", [0.5, 3.0])
def test_gradient_finite_differences(sigma):
    H, G = workloads.gauss(16, sigma, seed=34)
    H, G = H.astype(np.float64), G.astype(np.float64)
    n = 20
    dH = oracle.sk_bwd(H, G, n)
    h = 1e-6
    fd = np.zeros_like(H)
    for kl in range(16):
        k, l = divmod(kl, 4)
        E = np.zeros((4, 4))
        E[k, l] = h
        fd[:, k, l] = (G * (oracle.sk_fwd(H + E, n) - oracle.sk_fwd(H - E, n))).sum(axis=(1, 2)) / (2 * h)
    assert np.abs(dH - fd).max() < 1e-8 * max(1.0, np.abs(fd).max())


def test_gradient_autograd():
    H, G = workloads.gauss(64, 2.0, seed=35)
    Ht = torch.tensor(H, dtype=torch.float64, requires_grad=True)
    A = torch.exp(Ht)
    v = torch.ones(64, 4, dtype=torch.float64)
    for _ in range(20):
        u = 1.0 / (A @ v[..., None])[..., 0]
        v = 1.0 / (A.transpose(1, 2) @ u[..., None])[..., 0]
    P = u[..., :, None] * A * v[..., None, :]
    (P * torch.tensor(G, dtype=torch.float64)).sum().backward()
    assert np.abs(oracle.sk_bwd(H, G, 20) - Ht.grad.numpy()).max() < 1e-12
    assert np.abs(oracle.sk_fwd(H, 20) - P.detach().numpy()).max() < 1e-14
