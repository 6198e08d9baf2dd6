"""Full-size workloads, in the launch configuration the benchmark times.

Every matrix of every benchmark workload is compared with the oracle: P element by
element, the dual against its per-matrix conditioning bound, dH element by element,
and the marginals in fp64. The oracle runs chunk by chunk on the host threads.
"""
import time

import numpy as np
import pytest
import torch

import paper_2606_07574_amd as b4
import workloads
from tests._gpu import (GPU_TOL, MAX_ITER, TOL_DH, TOL_DH_SUMS, TOL_MARGINAL, TOL_P, bits_to_dev,
                        check_parity, dh_sums_rel_device, marginal_linf_device, parity_arrays, say,
                        to_dev)

pytestmark = pytest.mark.gpu

CHECK_CHUNK = 1 << 21  # matrices per oracle call (bounds the host memory of one comparison)


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


def _compare_all(name, ch, P, dual, dH):
    """Every matrix against the oracle; returns the running maxima."""
    B = ch.H.shape[0]
    worst = {"p_err": 0.0, "marg": 0.0, "dual_ratio": 0.0, "dh_err": 0.0, "kkt": 0.0}
    n_det, det_err = 0, 0.0
    t0 = time.time()
    for s in range(0, B, CHECK_CHUNK):
        e = min(B, s + CHECK_CHUNK)
        dPs = ch.dP[s:e] if dH is not None else None
        a = parity_arrays(ch.H[s:e], P[s:e].cpu().numpy(), dual[s:e].cpu().numpy(), dPs,
                          dH[s:e].cpu().numpy() if dH is not None else None)
        assert (a["oracle_iters"] >= 0).all(), f"{name}: oracle failed to converge in [{s}, {e})"
        assert (a["beta4"] == 0).all()
        ratio = a["dual_err"] / a["dual_bound"]
        det = a["dual_bound"] <= 1e-3
        n_det += int(det.sum())
        det_err = max(det_err, float(a["dual_err"][det].max()) if det.any() else 0.0)
        for k, v in (("p_err", a["p_err"]), ("marg", a["marg"]), ("dual_ratio", ratio), ("kkt", a["kkt"])):
            worst[k] = max(worst[k], float(v.max()))
        if dH is not None:
            worst["dh_err"] = max(worst["dh_err"], float(a["dh_err"].max()))
        if worst["p_err"] > TOL_P or worst["dual_ratio"] > 1.0 or worst["dh_err"] > TOL_DH:
            bad = int(np.argmax(a["p_err"])) + s
            say(f"  first failing chunk [{s}, {e}); worst P matrix {bad}")
            break
    say(f"  [{name}] all {B} matrices in {time.time() - t0:.1f}s: max|P-Pref|={worst['p_err']:.3e} "
        f"max marginal={worst['marg']:.3e} max dH rel err={worst['dh_err']:.3e}")
    say(f"  [{name}] dual: max err/bound={worst['dual_ratio']:.3f}; {n_det} of {B} determined "
        f"(bound <= 1e-3), max err there {det_err:.3e}; kkt rel err={worst['kkt']:.3e}")
    return worst


@pytest.mark.parametrize("name", ["n01_b2e20_fwd", "n10_b2e22", "mix_bf16_b2e24", "logunif_b2e25"])
def test_fullsize(name):
    say(f"test: full-size workload {name}, every matrix against the oracle")
    ch, Hd, dPd = _inputs(name)
    B = ch.H.shape[0]
    P, dual, it = b4.fwd(Hd, GPU_TOL, MAX_ITER, want_dual=True, want_iters=True)
    dH = b4.bwd(P, dPd) if dPd is not None else None
    torch.cuda.synchronize()
    itn = it.cpu().numpy()
    hist = np.bincount(np.clip(itn, 0, 64))
    say(f"  iters: mean={itn.mean():.3f} max={itn.max()} not_converged={(itn == -1).sum()} "
        f"hist(0..)={hist[:24].tolist()}")
    assert (itn >= 0).all()
    marg = marginal_linf_device(P)
    say(f"  max marginal over all {B} matrices (fp64 on the device): {marg.max().item():.3e}")
    assert marg.max().item() <= TOL_MARGINAL
    assert torch.isfinite(P).all()
    if dH is not None:
        assert torch.isfinite(dH).all()
        sums = dh_sums_rel_device(dH)
        say(f"  max |row/col sums of dH| / max(1, max|dH|): {sums.max().item():.2e}")
        assert sums.max().item() <= TOL_DH_SUMS
    worst = _compare_all(name, ch, P, dual, dH)
    assert worst["p_err"] <= TOL_P
    assert worst["marg"] <= TOL_MARGINAL
    assert worst["dual_ratio"] <= 1.0
    assert worst["kkt"] < 2e-4
    assert worst["dh_err"] <= TOL_DH


def test_beyond_32bit_offsets():
    # B = 2^27 fp32 matrices: every array is 8 GB (dual 4 GB) and byte offsets pass 2^32 at
    # b = 2^26; both forward variants' index arithmetic is 64-bit. Every matrix is checked for
    # convergence and marginals; parity on samples around 2^26 and at the end.
    B = 1 << 27
    say(f"test: B={B} fp32 (8 GB per array), throughput forward + backward")
    g = torch.Generator(device="cuda").manual_seed(27)
    H = 5.0 * torch.randn(B, 4, 4, device="cuda", generator=g)
    G = torch.randn(B, 4, 4, device="cuda", generator=g)
    P, dual, it = b4.fwd(H, GPU_TOL, MAX_ITER, want_dual=True, want_iters=True)
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
