"""GPU parity of the saved-Hessian variant (Sec. 4.2): birkhoff4_fwd_hess gives the same P and
dual as the one-problem-per-lane forward and the column weights of that P; birkhoff4_bwd_hess,
fed those weights, matches the oracle's backward to the same bar as the default backward."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_07574_amd as b4
import workloads
from tests._gpu import TOL_DH, bits_to_dev, dh_rel_err, say, to_dev

pytestmark = pytest.mark.gpu


def weights_fp64(P):
    P = P.astype(np.float64)
    pairs = [(0, 1), (0, 2), (0, 3), (1, 2), (1, 3), (2, 3)]
    return np.stack([(P[:, :, j] * P[:, :, k]).sum(axis=1) for j, k in pairs], axis=1)


def check(Hd, dPd, H, dP, label):
    P, dual, hess, it = b4.fwd_hess(Hd, want_iters=True)
    P0, dual0, it0 = b4.fwd(Hd, want_iters=True, variant=b4.THROUGHPUT)
    dH = b4.bwd_hess(P, hess, dPd)
    dH0 = b4.bwd(P, dPd)
    torch.cuda.synchronize()
    assert torch.equal(P, P0) and torch.equal(dual, dual0) and torch.equal(it, it0)
    Pn, hn = P.cpu().numpy(), hess.cpu().numpy()
    werr = np.abs(hn[:, :6] - weights_fp64(Pn)).max()
    assert (hn[:, 6:] == 0).all()
    ref = oracle.bwd(oracle.fwd(H)[0], dP)
    e = dh_rel_err(dH.cpu().numpy().astype(np.float64), ref).max()
    e0 = np.abs(dH.cpu().numpy() - dH0.cpu().numpy()).max() / max(1.0, np.abs(dH0.cpu().numpy()).max())
    say(f"  [{label}] max weight err={werr:.2e} dH rel err={e:.3e} vs default backward {e0:.2e}")
    assert werr <= 1e-6
    assert e <= TOL_DH


@pytest.mark.parametrize("sigma", [1.0, 10.0, 50.0])
def test_saved_hessian_parity(sigma):
    say(f"test: saved-Hessian variant, sigma={sigma}")
    H, dP = workloads.gauss(20011, sigma, seed=50 + int(sigma))
    check(to_dev(H), to_dev(dP), H, dP, f"sigma={sigma}")


def test_saved_hessian_bf16_mixture():
    say("test: saved-Hessian variant on the bf16 mixture")
    ch = workloads.make_chunk(workloads.WORKLOADS["mix_bf16_b2e24"], 0, B=1 << 16)
    check(bits_to_dev(ch.H_bits), bits_to_dev(ch.dP_bits), ch.H, ch.dP, "bf16 mix")


@pytest.mark.parametrize("B", [1, 63, 64, 65, 1000])
def test_saved_hessian_ragged(B):
    H, dP = workloads.gauss(B, 3.0, seed=B)
    check(to_dev(H), to_dev(dP), H, dP, f"B={B}")
