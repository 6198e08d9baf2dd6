"""GPU parity for n = 8: birkhoff8_fwd / birkhoff8_bwd against the size-generic fp64
oracle, element by element, with the same bars as the 4 x 4 path (max |P - P_ref| and
max marginal error <= 1e-5, per-matrix dH error <= 1e-4 relative to max(1, |dH_ref|)).
"""
import numpy as np
import pytest
import torch

import paper_2606_07574_amd as b4
from oracle import birkhoffn as on
import workloads
from tests._gpu import TOL_DH, TOL_MARGINAL, TOL_P, bits_to_dev, say, to_dev

pytestmark = pytest.mark.gpu

MAX_ITER = 64


def gauss8(B, sigma, seed):
    rng = np.random.default_rng(seed)
    H = (sigma * rng.standard_normal((B, 8, 8))).astype(np.float32)
    G = rng.standard_normal((B, 8, 8)).astype(np.float32)
    return H, G


def near_perm8(B, gap, noise, seed):
    rng = np.random.default_rng(seed)
    H = noise * rng.standard_normal((B, 8, 8))
    for b in range(B):
        H[b, np.arange(8), rng.permutation(8)] += gap
    return H.astype(np.float32)


def run(H, G=None, tol=1e-6, max_iter=MAX_ITER, dtype=torch.float32):
    Hd = to_dev(H) if dtype == torch.float32 else to_dev(H).to(torch.bfloat16)
    P, dual, it = b4.fwd8(Hd, tol, max_iter, want_dual=True, want_iters=True)
    dH = b4.bwd8(P, to_dev(G)) if G is not None else None
    torch.cuda.synchronize()
    return (P.cpu().numpy(), dual.cpu().numpy(), it.cpu().numpy(),
            None if dH is None else dH.cpu().numpy())


def check(H, P, dual, G=None, dH=None, label=""):
    Pr, _, itr = on.fwd(H.astype(np.float64))
    assert (itr >= 0).all(), f"{label}: oracle failed"
    perr = np.abs(P.astype(np.float64) - Pr).max()
    marg = on.marginal_errors(P).max()
    say(f"  [{label}] max|P-Pref|={perr:.3e} max marginal={marg:.3e}")
    assert perr <= TOL_P and marg <= TOL_MARGINAL
    if dual is not None:
        P64 = P.astype(np.float64)
        mask = P64 > 1e-4
        kkt = np.log(np.where(mask, P64, 1.0)) - H - dual[:, :8, None] - dual[:, None, 8:]
        scale = 1.0 + np.abs(H).max(axis=(1, 2), keepdims=True)
        kerr = (np.abs(kkt) / scale)[mask].max()
        say(f"  [{label}] dual kkt rel err={kerr:.3e}")
        assert kerr < 2e-4 and (dual[:, 15] == 0).all()
    if G is not None:
        ref = on.bwd(Pr, G.astype(np.float64)).reshape(-1, 64)
        e = np.abs(dH.reshape(-1, 64) - ref).max(axis=1) / np.maximum(1.0, np.abs(ref).max(axis=1))
        say(f"  [{label}] max dH rel err={e.max():.3e}")
        assert e.max() <= TOL_DH


@pytest.mark.parametrize("sigma", [0.1, 1.0, 5.0, 20.0, 50.0, 100.0])
def test_scales(sigma):
    say(f"test: n=8 gauss sigma={sigma}")
    H, G = gauss8(6000, sigma, seed=int(10 * sigma) + 1)
    P, dual, it, dH = run(H, G)
    say(f"  iters: mean={it.mean():.2f} max={it.max()} failed={(it < 0).sum()}")
    assert (it >= 0).all()
    check(H, P, dual, G, dH, f"sigma={sigma}")


# The forward's grid is the resident waves, each taking every nwv-th batch of 32 problems:
# batch counts below, at and above one batch per wave, and several batches per wave with a
# ragged last batch.
@pytest.mark.parametrize("B", [1, 2, 31, 32, 33, 63, 64, 65, 255, 257, 1000, 4097, 65535, 65569, 300007])
def test_ragged_batches(B):
    say(f"test: n=8 ragged B={B}")
    H, G = gauss8(B, 3.0, seed=B)
    P, dual, it, dH = run(H, G)
    assert (it >= 0).all()
    check(H, P, dual, G, dH, f"B={B}")


@pytest.mark.parametrize("gap,noise", [(20.0, 0.1), (8.0, 1.0), (3.0, 1.0), (60.0, 0.1)])
def test_near_permutations(gap, noise):
    say(f"test: n=8 near-permutations gap={gap} noise={noise}")
    H = near_perm8(5000, gap, noise, seed=int(gap + 10 * noise))
    G = np.random.default_rng(6).standard_normal(H.shape).astype(np.float32)
    P, dual, it, dH = run(H, G)
    say(f"  iters: mean={it.mean():.2f} max={it.max()} failed={(it < 0).sum()}")
    assert (it >= 0).all()
    check(H, P, dual, G, dH, "near-perm")


def test_bf16_storage():
    say("test: n=8 bf16 H and dP")
    H, G = gauss8(4000, 5.0, seed=9)
    Hb = torch.from_numpy(H).to(torch.bfloat16)
    Gb = torch.from_numpy(G).to(torch.bfloat16)
    P, dual, it = b4.fwd8(Hb.cuda(), want_dual=True, want_iters=True)
    dH = b4.bwd8(P, Gb.cuda())
    torch.cuda.synchronize()
    assert (it.cpu().numpy() >= 0).all()
    check(Hb.float().numpy(), P.cpu().numpy(), dual.cpu().numpy(), Gb.float().numpy(), dH.cpu().numpy(), "bf16")


def test_edge_cases():
    say("test: n=8 edge cases (B=0, non-finite, max_iter=0, separable)")
    P, dual, it = b4.fwd8(torch.empty(0, 8, 8, device="cuda"), want_iters=True)
    assert P.shape == (0, 8, 8)
    H, _ = gauss8(70, 2.0, seed=11)
    H[3, 2, 5] = np.nan
    H[68, 0, 0] = np.inf
    P, dual, it, _ = run(H)
    assert it[3] == b4.NON_FINITE and it[68] == b4.NON_FINITE
    assert np.isnan(P[3]).all() and np.isnan(P[68]).all()
    ok = np.setdiff1d(np.arange(70), [3, 68])
    assert (it[ok] >= 0).all()
    check(H[ok], P[ok], dual[ok], label="finite rows")
    P0, _, it0, _ = run(H[ok], max_iter=0)
    assert ((it0 == 0) | (it0 == b4.NOT_CONVERGED)).all()
    rng = np.random.default_rng(12)
    Hs = (5 * rng.standard_normal((64, 8, 1)) + 5 * rng.standard_normal((64, 1, 8))).astype(np.float32)
    Ps, _, its, _ = run(Hs)
    assert np.abs(Ps - 0.125).max() < 1e-5


def test_autograd_project8():
    say("test: n=8 autograd")
    H, G = gauss8(500, 4.0, seed=13)
    Hd = to_dev(H).requires_grad_(True)
    P = b4.project8(Hd)
    (P * to_dev(G)).sum().backward()
    torch.cuda.synchronize()
    check(H, P.detach().cpu().numpy(), None, G, Hd.grad.cpu().numpy(), "autograd")


def test_large_batch_sampled():
    B = 1 << 20
    say(f"test: n=8 B={B} sigma=5, sampled parity")
    H, G = gauss8(B, 5.0, seed=14)
    P, dual, it, dH = run(H, G)
    assert (it >= 0).all()
    marg = np.maximum(np.abs(P.astype(np.float64).sum(2) - 1).max(1), np.abs(P.astype(np.float64).sum(1) - 1).max(1))
    say(f"  iters mean={it.mean():.2f} max={it.max()}; max marginal over all {B}: {marg.max():.3e}")
    assert marg.max() <= TOL_MARGINAL
    idx = np.random.default_rng(15).choice(B, 3000, replace=False)
    check(H[idx], P[idx], dual[idx], G[idx], dH[idx], "sampled")


def test_fullsize_bench_workload():
    # the benchmark's 8x8 workload and launch (bf16 H and dP, dual written, no step counts);
    # a second launch with step counts must give the same bits
    B = 1 << 22
    say(f"test: n=8 full-size mixture B={B} (bf16), benchmark launch")
    H, G = workloads.n8_mix_device(B, 8, "cuda")
    P, dual, _ = b4.fwd8(H, 1e-6, MAX_ITER, want_dual=True)
    dH = b4.bwd8(P, G)
    P2, dual2, it = b4.fwd8(H, 1e-6, MAX_ITER, want_dual=True, want_iters=True)
    torch.cuda.synchronize()
    assert torch.equal(P, P2) and torch.equal(dual, dual2)
    itn = it.cpu().numpy()
    P64 = P.double()
    marg = torch.maximum((P64.sum(-1) - 1).abs().amax(-1), (P64.sum(-2) - 1).abs().amax(-1)).cpu().numpy()
    del P64, P2, dual2
    say(f"  iters mean={itn.mean():.2f} max={itn.max()} not converged={(itn < 0).sum()}; "
        f"max marginal over all {B}: {marg.max():.3e}")
    assert (itn >= 0).all()
    assert marg.max() <= TOL_MARGINAL
    rng = np.random.default_rng(16)
    idx = np.unique(np.concatenate([rng.choice(B, 3000, replace=False), np.argsort(marg)[-200:],
                                    np.argsort(itn)[-200:], np.arange(64), np.arange(B - 64, B)]))
    it_ = torch.from_numpy(idx).cuda()
    check(H[it_].float().cpu().numpy(), P[it_].cpu().numpy(), dual[it_].cpu().numpy(),
          G[it_].float().cpu().numpy(), dH[it_].cpu().numpy(), "full-size sample")
