"""GPU parity: the HIP path against the fp64 oracle, element by element.

Sizes here finish in seconds on the oracle, span many waves, and include
ragged tails; full-size workloads are in test_gpu_fullsize.py.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_07574_amd as b4
import workloads
from tests._gpu import (MAX_ITER, TOL_DH, TOL_P, VARIANT_IDS, VARIANTS, bits_to_dev, check_parity,
                        dh_rel_err, gpu_fwd, say, to_dev)

variants = pytest.mark.parametrize("variant", VARIANTS, ids=VARIANT_IDS)

pytestmark = pytest.mark.gpu


@variants
def test_n01_b4096_fwd_bwd(variant):
    say(f"test: n01_b4096 full parity (fwd + bwd), variant {variant}")
    ch = workloads.make_chunk(workloads.WORKLOADS["n01_b4096"], 0)
    Hd = to_dev(ch.H)
    P, dual, it = gpu_fwd(Hd, variant=variant)
    dH = b4.bwd(P, to_dev(ch.dP))
    torch.cuda.synchronize()
    it = it.cpu().numpy()
    say(f"  iters: mean={it.mean():.2f} max={it.max()}")
    assert (it >= 0).all()
    check_parity(ch.H, P.cpu().numpy(), dual.cpu().numpy(), ch.dP, dH.cpu().numpy(), "n01_b4096")


@variants
@pytest.mark.parametrize("B", [1, 2, 3, 15, 16, 17, 63, 64, 65, 255, 257, 1000, 4097, 20011])
def test_ragged_batches(B, variant):
    say(f"test: ragged B={B} variant {variant}")
    H, dP = workloads.gauss(B, 5.0, seed=B)
    P, dual, it = gpu_fwd(to_dev(H), variant=variant)
    dH = b4.bwd(P, to_dev(dP))
    torch.cuda.synchronize()
    assert (it.cpu().numpy() >= 0).all()
    check_parity(H, P.cpu().numpy(), dual.cpu().numpy(), dP, dH.cpu().numpy(), f"B={B}")


@variants
@pytest.mark.parametrize("sigma", [0.1, 1.0, 10.0, 20.0, 50.0])
def test_scales(sigma, variant):
    say(f"test: gauss sigma={sigma} variant {variant}")
    H, dP = workloads.gauss(30000, sigma, seed=7)
    P, dual, it = gpu_fwd(to_dev(H), variant=variant)
    dH = b4.bwd(P, to_dev(dP))
    torch.cuda.synchronize()
    itn = it.cpu().numpy()
    say(f"  iters: mean={itn.mean():.2f} max={itn.max()} failed={(itn < 0).sum()}")
    assert (itn >= 0).all()
    check_parity(H, P.cpu().numpy(), dual.cpu().numpy(), dP, dH.cpu().numpy(), f"sigma={sigma}")


@variants
def test_near_permutation(variant):
    say(f"test: near permutations 20 Pi + 0.1 N and 60 Pi + N, variant {variant}")
    for gap, noise in [(20.0, 0.1), (60.0, 1.0)]:
        H, dP = workloads.near_permutation(20000, gap, noise, seed=3)
        P, dual, it = gpu_fwd(to_dev(H), variant=variant)
        dH = b4.bwd(P, to_dev(dP))
        torch.cuda.synchronize()
        assert (it.cpu().numpy() >= 0).all()
        check_parity(H, P.cpu().numpy(), dual.cpu().numpy(), dP, dH.cpu().numpy(), f"perm gap={gap}")


@variants
def test_bf16_mixture(variant):
    say(f"test: bf16 mixture (workload mix_bf16_b2e24, first 2^17 matrices), variant {variant}")
    w = workloads.WORKLOADS["mix_bf16_b2e24"]
    ch = workloads.make_chunk(w, 0, B=1 << 17)
    Hd = bits_to_dev(ch.H_bits)
    dPd = bits_to_dev(ch.dP_bits)
    P, dual, it = gpu_fwd(Hd, variant=variant)
    dH = b4.bwd(P, dPd)
    torch.cuda.synchronize()
    itn = it.cpu().numpy()
    say(f"  iters: mean={itn.mean():.2f} max={itn.max()}")
    assert (itn >= 0).all()
    check_parity(ch.H, P.cpu().numpy(), dual.cpu().numpy(), ch.dP, dH.cpu().numpy(), "bf16 mix")


@variants
def test_fp32_and_bf16_paths_agree_on_same_values(variant):
    say(f"test: bf16 storage == fp32 storage of the same values, variant {variant}")
    w = workloads.WORKLOADS["mix_bf16_b2e24"]
    ch = workloads.make_chunk(w, 0, B=10000)
    P1, d1, i1 = gpu_fwd(bits_to_dev(ch.H_bits), variant=variant)
    P2, d2, i2 = gpu_fwd(to_dev(ch.H), variant=variant)
    assert torch.equal(P1, P2) and torch.equal(i1, i2)
    g1 = b4.bwd(P1, bits_to_dev(ch.dP_bits))
    g2 = b4.bwd(P1, to_dev(ch.dP))
    assert torch.equal(g1, g2)


@variants
def test_permutation_equivariance_on_gpu(variant):
    say(f"test: row/column permutation equivariance, variant {variant}")
    H, dP = workloads.gauss(5000, 8.0, seed=11)
    rng = np.random.default_rng(0)
    pr, pc = rng.permutation(4), rng.permutation(4)
    P, _, _ = gpu_fwd(to_dev(H), variant=variant)
    Pp, _, _ = gpu_fwd(to_dev(np.ascontiguousarray(H[:, pr][:, :, pc])), variant=variant)
    P = P.cpu().numpy()
    Pp = Pp.cpu().numpy()
    assert np.abs(Pp - P[:, pr][:, :, pc]).max() < 2e-6


def test_autograd_function():
    say("test: autograd Birkhoff4Fn")
    H, dP = workloads.gauss(3000, 3.0, seed=12)
    Hd = to_dev(H).requires_grad_(True)
    P = b4.project(Hd)
    (P * to_dev(dP)).sum().backward()
    ref = oracle.bwd(oracle.fwd(H)[0], dP)
    assert dh_rel_err(Hd.grad.cpu().numpy().astype(np.float64), ref).max() <= TOL_DH


@variants
def test_edge_cases(variant):
    say(f"test: edge cases (B=0, max_iter=0, tol=0, non-finite), variant {variant}")
    Z = torch.zeros(0, 4, 4, device="cuda:0")
    P, dual, it = b4.fwd(Z, want_iters=True, variant=variant)
    assert P.shape == (0, 4, 4)
    assert b4.bwd(P, Z).shape == (0, 4, 4)
    # max_iter = 0 returns T at the initial point: row softmax after column centring
    H, _ = workloads.gauss(500, 4.0, seed=13)
    P, dual, it = b4.fwd(to_dev(H), 1e-6, 0, want_iters=True, variant=variant)
    Hc = H.astype(np.float64) - H.astype(np.float64).mean(axis=1, keepdims=True)
    E = np.exp(Hc - Hc.max(axis=2, keepdims=True))
    ref = E / E.sum(axis=2, keepdims=True)
    itn = it.cpu().numpy()
    assert np.abs(P.cpu().numpy() - ref).max() < 2e-6
    conv0 = oracle.marginal_errors(ref)[0] <= 1e-6
    assert ((itn == 0) == conv0).all() and ((itn == -1) == ~conv0).all()
    # tol = 0: a matrix stops only when its fp32 column sums are exactly one, else
    # it runs to max_iter and is reported not converged; the result is still valid
    P, dual, it = b4.fwd(to_dev(H), 0.0, 7, want_iters=True, variant=variant)
    itn = it.cpu().numpy()
    assert ((itn == -1) | ((itn >= 0) & (itn <= 7))).all() and (itn == -1).any()
    assert np.abs(P.cpu().numpy().sum(axis=2) - 1).max() < 1e-5
    assert oracle.marginal_errors(P.cpu().numpy())[0].max() <= 1e-5
    # non-finite inputs poison only their own matrix
    H2, _ = workloads.gauss(300, 2.0, seed=14)
    H2[5, 1, 2] = np.nan
    H2[77, 0, 0] = np.inf
    H2[78, 3, 3] = -np.inf
    P, dual, it = b4.fwd(to_dev(H2), want_iters=True, variant=variant)
    Pn, itn, dn = P.cpu().numpy(), it.cpu().numpy(), dual.cpu().numpy()
    bad = [5, 77, 78]
    assert (itn[bad] == -2).all() and np.isnan(Pn[bad]).all() and np.isnan(dn[bad]).all()
    good = np.setdiff1d(np.arange(300), bad)
    assert (itn[good] >= 0).all()
    Pr = oracle.fwd(H2[good])[0]
    assert np.abs(Pn[good] - Pr).max() <= TOL_P


def test_batch_shapes_and_streams():
    say("test: leading batch dims and a side stream")
    H, dP = workloads.gauss(2 * 3 * 50, 2.0, seed=15)
    Hd = to_dev(H).reshape(2, 3, 50, 4, 4)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        P, dual, it = b4.fwd(Hd, want_iters=True)
        dH = b4.bwd(P, to_dev(dP).reshape(2, 3, 50, 4, 4))
    s.synchronize()
    assert P.shape == (2, 3, 50, 4, 4) and dual.shape == (2, 3, 50, 8) and it.shape == (2, 3, 50)
    check_parity(H, P.reshape(-1, 4, 4).cpu().numpy(), dual.reshape(-1, 8).cpu().numpy(), dP,
                 dH.reshape(-1, 4, 4).cpu().numpy(), "5-d batch")


@pytest.mark.parametrize("sigma", [0.5, 3.0])
def test_sinkhorn_baseline(sigma):
    say(f"test: SK-20 baseline sigma={sigma}")
    H, dP = workloads.gauss(20000, sigma, seed=16)
    P = b4.sk_fwd(to_dev(H), 20)
    dH = b4.sk_bwd(to_dev(H), to_dev(dP), 20)
    torch.cuda.synchronize()
    Pr = oracle.sk_fwd(H, 20)
    dHr = oracle.sk_bwd(H, dP, 20)
    assert np.abs(P.cpu().numpy() - Pr).max() <= 1e-5
    assert dh_rel_err(dH.cpu().numpy().astype(np.float64), dHr).max() <= TOL_DH
    # columns of the SK output sum to one after the final column step
    assert np.abs(P.cpu().numpy().astype(np.float64).sum(axis=1) - 1).max() < 2e-6


@pytest.mark.parametrize("n_steps", [1, 7, 19, 21, 48])
def test_sinkhorn_step_counts(n_steps):
    # 20 steps run the register-resident backward; every other count the LDS one
    say(f"test: SK-{n_steps} baseline")
    H, dP = workloads.gauss(5000, 3.0, seed=30 + n_steps)
    P = b4.sk_fwd(to_dev(H), n_steps)
    dH = b4.sk_bwd(to_dev(H), to_dev(dP), n_steps)
    torch.cuda.synchronize()
    assert np.abs(P.cpu().numpy() - oracle.sk_fwd(H, n_steps)).max() <= 1e-5
    assert dh_rel_err(dH.cpu().numpy().astype(np.float64), oracle.sk_bwd(H, dP, n_steps)).max() <= TOL_DH


def test_sinkhorn_bf16():
    say("test: SK-20 baseline on bf16 H and dP")
    ch = workloads.make_chunk(workloads.WORKLOADS["mix_bf16_b2e24"], 0, B=20000)
    Hd, dPd = bits_to_dev(ch.H_bits), bits_to_dev(ch.dP_bits)
    P = b4.sk_fwd(Hd, 20)
    dH = b4.sk_bwd(Hd, dPd, 20)
    torch.cuda.synchronize()
    assert np.abs(P.cpu().numpy() - oracle.sk_fwd(ch.H, 20)).max() <= 1e-5
    assert dh_rel_err(dH.cpu().numpy().astype(np.float64), oracle.sk_bwd(ch.H, ch.dP, 20)).max() <= TOL_DH


def test_variants_agree():
    say("test: throughput and latency variants give the same projection")
    H, _ = workloads.gauss(50000, 6.0, seed=21)
    Hd = to_dev(H)
    P1, d1, i1 = gpu_fwd(Hd, variant=b4.THROUGHPUT)
    P2, d2, i2 = gpu_fwd(Hd, variant=b4.LATENCY)
    diff = (P1 - P2).abs().max().item()
    say(f"  max |P_throughput - P_latency| = {diff:.2e}")
    assert diff <= 2 * TOL_P
    assert (i1 >= 0).all() and (i2 >= 0).all()


def test_binding_rejects_mismatched_outputs():
    say("test: binding rejects an out tensor the kernel could overrun")
    H = to_dev(workloads.gauss(100, 1.0, seed=40)[0])
    for bad in (torch.empty(99, 4, 4, device="cuda"), torch.empty(100, 4, 4, device="cuda", dtype=torch.float16),
                torch.empty(100, 4, 8, device="cuda")[..., ::2]):
        with pytest.raises(ValueError):
            b4.fwd(H, out=bad)
    P, _, _ = b4.fwd(H)
    with pytest.raises(ValueError):
        b4.bwd(P, H, out=torch.empty(50, 4, 4, device="cuda"))
    with pytest.raises(ValueError):
        b4.fwd8(torch.zeros(10, 8, 8, device="cuda"), out=torch.empty(10, 4, 4, device="cuda"))


@pytest.mark.parametrize("B", [1000, 100003])
def test_plain_signatures(B):
    # birkhoff4_fwd(H, P, dual, B, tol, max_iter, stream) and birkhoff4_bwd(P, dual, dP, dH, B,
    # stream) called directly through the C ABI on device buffers (fp32, the default dispatch:
    # the four-lanes-per-problem forward below 2^15 problems, the throughput forward above)
    say(f"test: birkhoff4_fwd / birkhoff4_bwd through the C ABI, B={B}")
    H, dP = workloads.gauss(B, 5.0, seed=B + 17)
    Hd, dPd = to_dev(H), to_dev(dP)
    P = torch.empty(B, 4, 4, device="cuda:0")
    dual = torch.empty(B, 8, device="cuda:0")
    dH = torch.empty(B, 4, 4, device="cuda:0")
    lib = b4.lib()
    stream = torch.cuda.current_stream().cuda_stream
    assert lib.birkhoff4_fwd(Hd.data_ptr(), P.data_ptr(), dual.data_ptr(), B, 1e-6, MAX_ITER, stream) == 0
    assert lib.birkhoff4_bwd(P.data_ptr(), dual.data_ptr(), dPd.data_ptr(), dH.data_ptr(), B, stream) == 0
    torch.cuda.synchronize()
    check_parity(H, P.cpu().numpy(), dual.cpu().numpy(), dP, dH.cpu().numpy(), f"C ABI B={B}")
    # the backward accepts dual = NULL (it reads only P and dP) and gives the same dH
    dH2 = torch.empty_like(dH)
    assert lib.birkhoff4_bwd(P.data_ptr(), None, dPd.data_ptr(), dH2.data_ptr(), B, stream) == 0
    torch.cuda.synchronize()
    assert torch.equal(dH, dH2)
