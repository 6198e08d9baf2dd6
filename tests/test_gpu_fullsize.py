"""Full-size workloads, in the launch configuration the benchmark times.

Every matrix is checked for convergence and for its marginal error (fp64 sums
on the device); P, dual and dH parity with the oracle is checked on a sample
the oracle can afford: random indices plus the matrices with the largest
marginal error and the most Newton steps.
"""
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2606_07574_amd as b4
import workloads
from tests._gpu import (MAX_ITER, TOL_MARGINAL, bits_to_dev, check_parity, marginal_linf_device,
                        say, to_dev)

pytestmark = pytest.mark.gpu


def _inputs(name):
    t0 = time.time()
    ch = workloads.generate(name, threads=16)
    say(f"  generated {name}: B={ch.H.shape[0]} in {time.time() - t0:.1f}s")
    if ch.H_bits is not None:
        Hd = bits_to_dev(ch.H_bits)
        dPd = bits_to_dev(ch.dP_bits) if ch.dP_bits is not None else None
    else:
        Hd = to_dev(ch.H)
        dPd = to_dev(ch.dP) if ch.dP is not None else None
    return ch, Hd, dPd


def _sample(B, marg, it, k=4096, seed=0):
    rng = np.random.default_rng(seed)
    idx = set(rng.choice(B, size=min(k, B), replace=False).tolist())
    idx |= set(np.argsort(marg)[-256:].tolist())
    idx |= set(np.argsort(it)[-256:].tolist())
    idx |= set(range(min(64, B))) | set(range(max(0, B - 64), B))
    return np.array(sorted(idx))


@pytest.mark.parametrize("name", ["n01_b2e20_fwd", "n10_b2e22", "mix_bf16_b2e24", "logunif_b2e25"])
def test_fullsize(name):
    say(f"test: full-size workload {name}")
    ch, Hd, dPd = _inputs(name)
    B = ch.H.shape[0]
    P, dual, it = b4.fwd(Hd, 1e-6, MAX_ITER, want_dual=True, want_iters=True)
    dH = b4.bwd(P, dPd) if dPd is not None else None
    torch.cuda.synchronize()
    itn = it.cpu().numpy()
    marg = marginal_linf_device(P).cpu().numpy()
    hist = np.bincount(np.clip(itn, 0, 64))
    say(f"  iters: mean={itn.mean():.3f} max={itn.max()} not_converged={(itn == -1).sum()} "
        f"hist(0..)={hist[:24].tolist()}")
    say(f"  max marginal over all {B} matrices: {marg.max():.3e}")
    assert (itn >= 0).all()
    assert marg.max() <= TOL_MARGINAL
    assert torch.isfinite(P).all()
    if dH is not None:
        assert torch.isfinite(dH).all()
        # row and column sums of dH vanish for every matrix, up to rounding
        d64 = dH.double()
        sums = torch.maximum(d64.sum(dim=-1).abs().amax(dim=-1), d64.sum(dim=-2).abs().amax(dim=-1))
        worst = int(torch.argmax(sums).item())
        say(f"  max |row/col sums of dH|: {sums[worst].item():.2e} at matrix {worst}, "
            f"max|dH| there {dH[worst].abs().max().item():.3e}")
        worst_ix = np.array([worst])
        check_parity(ch.H[worst_ix], P[worst:worst + 1].cpu().numpy(), None,
                     ch.dP[worst_ix], dH[worst:worst + 1].cpu().numpy(), f"{name} worst dH sums")
        assert sums.max().item() < 1e-4
    idx = _sample(B, marg, itn)
    idx_t = torch.from_numpy(idx).to("cuda:0")
    Ps = P[idx_t].cpu().numpy()
    ds = dual[idx_t].cpu().numpy()
    dHs = dH[idx_t].cpu().numpy() if dH is not None else None
    dPs = ch.dP[idx] if ch.dP is not None else None
    check_parity(ch.H[idx], Ps, ds, dPs, dHs, f"{name} sample of {len(idx)}")
