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


def test_beyond_32bit_offsets():
    # B = 2^27 fp32 matrices: every array is 8 GB (dual 4 GB) and byte offsets pass 2^32 at
    # b = 2^26; both forward variants' index arithmetic is 64-bit. Every matrix is checked for
    # convergence and marginals; parity on samples around 2^26 and at the end.
    B = 1 << 27
    say(f"test: B={B} fp32 (8 GB per array), throughput forward + backward")
    g = torch.Generator(device="cuda").manual_seed(27)
    H = 5.0 * torch.randn(B, 4, 4, device="cuda", generator=g)
    G = torch.randn(B, 4, 4, device="cuda", generator=g)
    P, dual, it = b4.fwd(H, 1e-6, MAX_ITER, want_dual=True, want_iters=True)
    dH = b4.bwd(P, G)
    torch.cuda.synchronize()
    assert (it >= 0).all().item()
    worst = 0.0
    for s in range(0, B, 1 << 24):  # fp64 marginals in slices, to bound the temporary memory
        worst = max(worst, marginal_linf_device(P[s:s + (1 << 24)]).max().item())
    say(f"  max marginal over all {B}: {worst:.3e}")
    assert worst <= TOL_MARGINAL
    rng = np.random.default_rng(27)
    idx = np.unique(np.concatenate([np.arange((1 << 26) - 64, (1 << 26) + 64), np.arange(B - 128, B),
                                    rng.choice(B, 1000, replace=False)]))
    ti = torch.from_numpy(idx).cuda()
    check_parity(H[ti].cpu().numpy(), P[ti].cpu().numpy(), dual[ti].cpu().numpy(), G[ti].cpu().numpy(),
                 dH[ti].cpu().numpy(), "B=2^27 sample")
