"""GPU parity for general entropic OT (4 x 4): birkhoff4_ot_fwd / birkhoff4_ot_bwd against the
fp64 OT oracle, element by element. Bars: max |T - T_ref| <= 1e-5 max(1, max a), column
marginals within 1e-5 of b, per-matrix dM error <= 1e-4 relative to max(1, |dM_ref|_inf).
"""
import numpy as np
import pytest
import torch

import paper_2606_07574_amd as b4
from oracle import birkhoffn as on
import workloads
from tests._gpu import say, to_dev

pytestmark = pytest.mark.gpu

TOL_T = 1e-5
TOL_MARG = 1e-5
TOL_DM = 1e-4


def problem(B, scale, seed, amin=0.2, amax=2.0):
    rng = np.random.default_rng(seed)
    M = (scale * rng.standard_normal((B, 4, 4))).astype(np.float32)
    a = rng.uniform(amin, amax, (B, 4)).astype(np.float32)
    b = rng.uniform(amin, amax, (B, 4))
    b = (b * (a.astype(np.float64).sum(1) / b.sum(1))[:, None]).astype(np.float32)
    G = rng.standard_normal((B, 4, 4)).astype(np.float32)
    return M, a, b, G


def run(M, a, b, eta, G=None, tol=1e-6, max_iter=64):
    T, dual, it = b4.ot_fwd(to_dev(M), to_dev(a), to_dev(b), eta, tol, max_iter, want_dual=True, want_iters=True)
    dM = b4.ot_bwd(T, to_dev(a), to_dev(G), eta) if G is not None else None
    torch.cuda.synchronize()
    return (T.cpu().numpy(), dual.cpu().numpy(), it.cpu().numpy(), None if dM is None else dM.cpu().numpy())


def check(M, a, b, eta, T, dual, G=None, dM=None, label=""):
    # the oracle sees the fp32 inputs as given (b's sums equal a's only to fp32 rounding)
    a64, b64 = a.astype(np.float64), b.astype(np.float64)
    b64 = b64 * (a64.sum(1) / b64.sum(1))[:, None]
    Tr, _, itr = on.ot_fwd(M.astype(np.float64), a64, b64, eta)
    assert (itr >= 0).all(), f"{label}: oracle failed"
    scale = np.maximum(1.0, a64.max(axis=1))[:, None, None]
    terr = (np.abs(T - Tr) / scale).max()
    cerr = np.abs(T.astype(np.float64).sum(1) - b64).max()
    rerr = np.abs(T.astype(np.float64).sum(2) - a64).max()
    say(f"  [{label}] max|T-Tref|/scale={terr:.3e} col marginal={cerr:.3e} row marginal={rerr:.3e}")
    assert terr <= TOL_T and cerr <= TOL_MARG and rerr <= TOL_MARG
    if dual is not None:
        T64 = T.astype(np.float64)
        mask = T64 > 1e-4 * scale
        kkt = eta * np.log(np.where(mask, T64, 1.0)) - (dual[:, :4, None] + dual[:, None, 4:] - M)
        rel = np.abs(kkt) / (eta + np.abs(M).max(axis=(1, 2), keepdims=True))
        kerr = rel[mask].max()
        say(f"  [{label}] dual kkt rel err={kerr:.3e}")
        assert kerr < 2e-4 and (dual[:, 7] == 0).all()
    if G is not None:
        ref = on.ot_bwd(Tr, a64, G.astype(np.float64), eta).reshape(-1, 16)
        e = np.abs(dM.reshape(-1, 16) - ref).max(axis=1) / np.maximum(1.0, np.abs(ref).max(axis=1))
        say(f"  [{label}] max dM rel err={e.max():.3e}")
        assert e.max() <= TOL_DM


@pytest.mark.parametrize("eta,scale", [(1.0, 1.0), (1.0, 5.0), (0.1, 2.0), (0.05, 1.0), (5.0, 20.0), (0.5, 10.0)])
def test_parity(eta, scale):
    say(f"test: OT eta={eta} cost scale={scale}")
    M, a, b, G = problem(20000, scale, seed=int(100 * eta + scale))
    T, dual, it, dM = run(M, a, b, eta, G)
    say(f"  iters mean={it.mean():.2f} max={it.max()} failed={(it < 0).sum()}")
    assert (it >= 0).all()
    check(M, a, b, eta, T, dual, G, dM, f"eta={eta}")


@pytest.mark.parametrize("eta,scale", [(0.1, 1.0), (0.5, 2.0), (0.1, 5.0), (0.02, 1.0)])
def test_wide_marginals(eta, scale):
    # a and b log-uniform over three decades (1e-3 .. 1), so rows and columns of T differ in
    # mass by up to 1000x; cost over eta reaches logit scales of 50
    say(f"test: OT marginals over three decades, eta={eta} cost scale={scale}")
    rng = np.random.default_rng(int(1000 * eta + scale))
    B = 20000
    M = (scale * rng.standard_normal((B, 4, 4))).astype(np.float32)
    a = np.exp(rng.uniform(np.log(1e-3), 0.0, (B, 4))).astype(np.float32)
    b = np.exp(rng.uniform(np.log(1e-3), 0.0, (B, 4)))
    b = (b * (a.astype(np.float64).sum(1) / b.sum(1))[:, None]).astype(np.float32)
    G = rng.standard_normal((B, 4, 4)).astype(np.float32)
    T, dual, it, dM = run(M, a, b, eta, G, max_iter=256)
    say(f"  iters mean={it.mean():.2f} max={it.max()} failed={(it < 0).sum()}")
    assert (it >= 0).all()
    check(M, a, b, eta, T, dual, G, dM, f"wide eta={eta}")


def test_birkhoff_special_case():
    say("test: OT with M = -H, a = b = 1, eta = 1 reproduces the projection")
    rng = np.random.default_rng(3)
    H = (5 * rng.standard_normal((5000, 4, 4))).astype(np.float32)
    G = rng.standard_normal(H.shape).astype(np.float32)
    ones = np.ones((5000, 4), np.float32)
    T, dual, it, dM = run(-H, ones, ones, 1.0, G)
    P, _, _ = b4.fwd(to_dev(H))
    dH = b4.bwd(P, to_dev(G))
    torch.cuda.synchronize()
    assert (it >= 0).all()
    assert np.abs(T - P.cpu().numpy()).max() < 2e-5
    assert np.abs(dM + dH.cpu().numpy()).max() / max(1.0, np.abs(dH.cpu().numpy()).max()) < 1e-4
    check(-H, ones, ones, 1.0, T, dual, G, dM, "birkhoff")


def test_separable_cost():
    say("test: OT separable cost gives a b^T / sum(a)")
    rng = np.random.default_rng(4)
    B = 3000
    M = (3 * rng.standard_normal((B, 4, 1)) + 3 * rng.standard_normal((B, 1, 4))).astype(np.float32)
    a = rng.uniform(0.5, 3.0, (B, 4)).astype(np.float32)
    b = rng.uniform(0.5, 3.0, (B, 4))
    b = (b * (a.astype(np.float64).sum(1) / b.sum(1))[:, None]).astype(np.float32)
    T, _, it, _ = run(M, a, b, 0.7)
    expect = a[:, :, None].astype(np.float64) * b[:, None, :] / a.astype(np.float64).sum(1)[:, None, None]
    assert (it >= 0).all()
    assert np.abs(T - expect).max() < 1e-5


# batch counts below, at and above one 64-problem batch per resident wave, and several per wave
@pytest.mark.parametrize("B", [1, 63, 64, 65, 1000, 70001, 131072, 300007])
def test_ragged(B):
    say(f"test: OT ragged B={B}")
    M, a, b, G = problem(B, 3.0, seed=B)
    T, dual, it, dM = run(M, a, b, 0.8, G)
    assert (it >= 0).all()
    check(M, a, b, 0.8, T, dual, G, dM, f"B={B}")


def test_edge_cases():
    say("test: OT edge cases (B=0, non-finite and non-positive inputs)")
    z = torch.empty(0, 4, 4, device="cuda")
    zv = torch.empty(0, 4, device="cuda")
    T, _, _ = b4.ot_fwd(z, zv, zv, 1.0)
    assert T.shape == (0, 4, 4)
    M, a, b, _ = problem(50, 2.0, seed=7)
    M[3, 1, 2] = np.nan
    a[10, 0] = 0.0
    b[20, 3] = -1.0
    M[30, 0, 0] = np.inf
    T, dual, it, _ = run(M, a, b, 1.0)
    bad = [3, 10, 20, 30]
    assert (it[bad] == b4.NON_FINITE).all()
    assert np.isnan(T[bad]).all()
    ok = np.setdiff1d(np.arange(50), bad)
    assert (it[ok] >= 0).all()
    check(M[ok], a[ok], b[ok], 1.0, T[ok], dual[ok], label="valid rows")


def test_autograd():
    say("test: OT autograd")
    M, a, b, G = problem(800, 2.0, seed=9)
    Md = to_dev(M).requires_grad_(True)
    T = b4.ot(Md, to_dev(a), to_dev(b), 0.6)
    (T * to_dev(G)).sum().backward()
    torch.cuda.synchronize()
    check(M, a, b, 0.6, T.detach().cpu().numpy(), None, G, Md.grad.cpu().numpy(), "autograd")


def test_fullsize_bench_workload():
    # the benchmark's OT workload and launch (dual written, no step counts); a second launch
    # with step counts must give the same bits
    B = 1 << 22
    say(f"test: OT full-size workload B={B}, benchmark launch")
    M, a, b, G = workloads.ot_device(B, 4, "cuda")
    T, dual, _ = b4.ot_fwd(M, a, b, 0.5, 1e-6, 64, want_dual=True)
    dM = b4.ot_bwd(T, a, G, 0.5)
    T2, dual2, it = b4.ot_fwd(M, a, b, 0.5, 1e-6, 64, want_dual=True, want_iters=True)
    torch.cuda.synchronize()
    assert torch.equal(T, T2) and torch.equal(dual, dual2)
    itn = it.cpu().numpy()
    T64 = T.double()
    marg = torch.maximum((T64.sum(-1) - a.double()).abs().amax(-1),
                         (T64.sum(-2) - b.double()).abs().amax(-1)).cpu().numpy()
    del T64, T2, dual2
    say(f"  iters mean={itn.mean():.2f} max={itn.max()} not converged={(itn < 0).sum()}; "
        f"max marginal over all {B}: {marg.max():.3e}")
    assert (itn >= 0).all()
    assert marg.max() <= TOL_MARG
    rng = np.random.default_rng(17)
    idx = np.unique(np.concatenate([rng.choice(B, 3000, replace=False), np.argsort(marg)[-200:],
                                    np.argsort(itn)[-200:], np.arange(64), np.arange(B - 64, B)]))
    it_ = torch.from_numpy(idx).cuda()
    check(M[it_].cpu().numpy(), a[it_].cpu().numpy(), b[it_].cpu().numpy(), 0.5, T[it_].cpu().numpy(),
          dual[it_].cpu().numpy(), G[it_].cpu().numpy(), dM[it_].cpu().numpy(), "full-size sample")
