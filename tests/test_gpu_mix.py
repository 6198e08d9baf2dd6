"""GPU parity of the residual-mixing pair (birkhoff4_mix_fwd / birkhoff4_mix_bwd, Sec. 2.1)
with the fp64 oracle, element by element.

Bounds, per element: P within 1e-5 of the oracle's (the projection's own bound), so an
output mixed from four inputs may differ by 1e-5 times the sum of their magnitudes, plus
fp32 rounding, plus for bf16 outputs one rounding to nearest even of the fp32 result. With an
8-bit significand, half a unit in the last place is at most 2^-8 of the value rounded, and that
value (the fp32 result) is within the additive slack of the exact one: 2^-8 (|ref| + slack) is
allowed, half of what a truncating conversion could reach. dH is held to the projection backward's bound,
|dH - dH_ref|_inf / max(1, |dH_ref|_inf) <= 1e-4 per token.
"""
import numpy as np
import pytest
import torch

import paper_2606_07574_amd as b4
import workloads
from oracle.mix import mix_bwd as o_bwd
from oracle.mix import mix_fwd as o_fwd
from tests._gpu import TOL_DH, TOL_P, say, to_dev

pytestmark = pytest.mark.gpu


def streams(B, C, seed, bf16):
    """X, dY ~ N(0,1) [B, 4, C] as fp32 arrays holding the values the GPU sees."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 77]))
    X = rng.standard_normal((B, 4, C), dtype=np.float32)
    G = rng.standard_normal((B, 4, C), dtype=np.float32)
    if bf16:
        X = workloads.bf16_to_f32(workloads.bf16_bits(X))
        G = workloads.bf16_to_f32(workloads.bf16_bits(G))
    return X, G


def mixed_bound(P_err, inputs, out_ref, bf16):
    """Per-element bound for an output mixed from the four streams of `inputs`."""
    s = np.abs(inputs).sum(axis=1, keepdims=True)
    b = P_err * s + 1e-6 * s + 1e-30
    if bf16:
        b = b + 2.0 ** -8 * (np.abs(out_ref) + b)
    return b


def check_case(H, X, G, dtype, label, h_dtype=torch.float32):
    bf16 = dtype == torch.bfloat16
    n = H.shape[-1]
    mfwd, mbwd = (b4.mix_fwd, b4.mix_bwd) if n == 4 else (b4.mix8_fwd, b4.mix8_bwd)
    Hd, Xd, Gd = to_dev(H, h_dtype), to_dev(X, dtype), to_dev(G, dtype)
    Y, P, _, it = mfwd(Hd, Xd, want_iters=True)
    dX, dH = mbwd(P, Xd, Gd)
    P_alone, _, _ = (b4.fwd if n == 4 else b4.fwd8)(Hd, want_dual=False)
    torch.cuda.synchronize()
    assert torch.equal(P, P_alone), f"{label}: P differs from the projection's own"
    assert (it.cpu().numpy() >= 0).all()
    Hh = Hd.float().cpu().numpy().astype(np.float64)
    Yr, Pr = o_fwd(Hh, X)
    dXr, dHr = o_bwd(Pr, X, G)
    Pg = P.cpu().numpy().astype(np.float64)
    perr = np.abs(Pg - Pr).max()
    assert perr <= TOL_P, f"{label}: max|P - P_ref| = {perr}"
    if X.shape[-1] > 0:
        Yg = Y.float().cpu().numpy().astype(np.float64)
        dXg = dX.float().cpu().numpy().astype(np.float64)
        ey = np.abs(Yg - Yr) / mixed_bound(TOL_P, X, Yr, bf16)
        ex = np.abs(dXg - dXr) / mixed_bound(TOL_P, G, dXr, bf16)
        say(f"  [{label}] max|P-Pref|={perr:.2e} Y err/bound={ey.max():.3f} dX err/bound={ex.max():.3f}")
        assert ey.max() <= 1.0, f"{label}: Y outside its bound"
        assert ex.max() <= 1.0, f"{label}: dX outside its bound"
    dHg = dH.cpu().numpy().astype(np.float64)
    e = np.abs(dHg - dHr).max(axis=(1, 2)) / np.maximum(1.0, np.abs(dHr).max(axis=(1, 2)))
    say(f"  [{label}] max dH rel err={e.max():.2e}")
    assert e.max() <= TOL_DH, f"{label}: dH rel err {e.max()}"


CASES = [  # B, C, stream dtype, logit scale
    (1, 8, torch.bfloat16, 1.0),
    (7, 24, torch.bfloat16, 5.0),
    (300, 520, torch.bfloat16, 5.0),     # 65 chunks per row: a full pass and a ragged one
    (300, 1032, torch.float32, 5.0),     # 258 chunks per row
    (257, 64, torch.float32, 20.0),
    (1000, 4096, torch.bfloat16, 1.0),
    (4099, 512, torch.bfloat16, 20.0),
    (33000, 16, torch.bfloat16, 5.0),    # beyond 32768 tokens: the throughput projection
    (64, 0, torch.bfloat16, 5.0),        # no channels: P and dH only (dH = 0)
]


@pytest.mark.parametrize("B,C,dtype,sigma", CASES,
                         ids=[f"B{b}-C{c}-{str(d)[6:]}-s{s:g}" for b, c, d, s in CASES])
def test_parity(B, C, dtype, sigma):
    say(f"test: mix parity B={B} C={C} {dtype} sigma={sigma}")
    H, _ = workloads.gauss(B, sigma, seed=B + C)
    X, G = streams(B, C, B * 7 + C, dtype == torch.bfloat16)
    check_case(H, X, G, dtype, f"B={B} C={C}")


def test_bf16_logits():
    say("test: mix with bf16 logits")
    H, _ = workloads.gauss(500, 5.0, seed=3)
    H = workloads.bf16_to_f32(workloads.bf16_bits(H))
    X, G = streams(500, 256, 4, True)
    check_case(H, X, G, torch.bfloat16, "bf16 H", h_dtype=torch.bfloat16)


def test_near_permutations_permute_streams():
    say("test: mix of near-permutation logits")
    H, _ = workloads.near_permutation(2000, 20.0, 0.1, seed=5)
    X, G = streams(2000, 128, 6, False)
    check_case(H, X, G, torch.float32, "near-permutation")


def test_non_finite_token():
    # a NaN logit poisons only its own token: NaN P, Y, dX and dH there, the others exact
    say("test: mix with a non-finite token")
    H, _ = workloads.gauss(100, 2.0, seed=8)
    H[17, 2, 1] = np.nan
    X, G = streams(100, 64, 9, True)
    Hd, Xd, Gd = to_dev(H), to_dev(X, torch.bfloat16), to_dev(G, torch.bfloat16)
    Y, P, _, it = b4.mix_fwd(Hd, Xd, want_iters=True)
    dX, dH = b4.mix_bwd(P, Xd, Gd)
    torch.cuda.synchronize()
    assert it[17].item() == b4.NON_FINITE
    for t in (Y, dX, dH, P):
        assert torch.isnan(t[17].float()).all()
        rest = torch.cat([t[:17], t[18:]]).float()
        assert torch.isfinite(rest).all()
    keep = np.r_[0:17, 18:100]
    check_case(H[keep], X[keep], G[keep], torch.bfloat16, "other tokens")


def test_empty_batch():
    Hd = torch.empty(0, 4, 4, device="cuda")
    Xd = torch.empty(0, 4, 64, device="cuda", dtype=torch.bfloat16)
    Y, P, _, _ = b4.mix_fwd(Hd, Xd)
    dX, dH = b4.mix_bwd(P, Xd, Xd)
    torch.cuda.synchronize()
    assert Y.shape == (0, 4, 64) and dH.shape == (0, 4, 4)


def test_leading_dims_and_autograd():
    say("test: mix autograd with leading dims")
    g = torch.Generator(device="cuda").manual_seed(12)
    H = (3.0 * torch.randn(6, 50, 4, 4, device="cuda", generator=g)).requires_grad_()
    X = torch.randn(6, 50, 4, 96, device="cuda", generator=g, dtype=torch.float32).to(torch.bfloat16)
    X.requires_grad_()
    W = torch.randn(6, 50, 4, 96, device="cuda", generator=g)
    Y = b4.mix(H, X)
    (Y.float() * W).sum().backward()
    Y2, P, _, _ = b4.mix_fwd(H.detach(), X.detach())
    dX, dH = b4.mix_bwd(P, X.detach(), W.to(torch.bfloat16))
    torch.cuda.synchronize()
    assert torch.equal(Y, Y2)
    assert torch.equal(H.grad, dH) and torch.equal(X.grad, dX)
    check_case(H.detach().reshape(-1, 4, 4).cpu().numpy(), X.detach().float().reshape(-1, 4, 96).cpu().numpy(),
               W.to(torch.bfloat16).float().reshape(-1, 4, 96).cpu().numpy(), torch.bfloat16, "leading dims")


def test_fullsize_bench_workload():
    # the benchmark's mixing workload and launch, checked on a sample of tokens
    B, C = 1 << 15, 4096
    say(f"test: mix full-size B={B} C={C} bf16, sampled")
    H, X, G = workloads.mix_streams_device(B, C, 60, "cuda")
    Y, P, _, it = b4.mix_fwd(H, X, want_iters=True)
    dX, dH = b4.mix_bwd(P, X, G)
    torch.cuda.synchronize()
    itn = it.cpu().numpy()
    say(f"  iters mean={itn.mean():.2f} max={itn.max()}")
    assert (itn >= 0).all()
    assert torch.isfinite(Y.float()).all() and torch.isfinite(dX.float()).all() and torch.isfinite(dH).all()
    idx = np.unique(np.concatenate([np.random.default_rng(3).choice(B, 200, replace=False),
                                    np.argsort(itn)[-20:], [0, B - 1]]))
    ti = torch.from_numpy(idx).cuda()
    Hs = H[ti].float().cpu().numpy()
    Xs = X[ti].float().cpu().numpy()
    Gs = G[ti].float().cpu().numpy()
    Yr, Pr = o_fwd(Hs, Xs)
    dXr, dHr = o_bwd(Pr, Xs, Gs)
    assert np.abs(P[ti].cpu().numpy() - Pr).max() <= TOL_P
    ey = np.abs(Y[ti].float().cpu().numpy() - Yr) / mixed_bound(TOL_P, Xs, Yr, True)
    ex = np.abs(dX[ti].float().cpu().numpy() - dXr) / mixed_bound(TOL_P, Gs, dXr, True)
    e = np.abs(dH[ti].cpu().numpy() - dHr).max(axis=(1, 2)) / np.maximum(1.0, np.abs(dHr).max(axis=(1, 2)))
    say(f"  sample of {len(idx)}: Y err/bound={ey.max():.3f} dX err/bound={ex.max():.3f} dH rel={e.max():.2e}")
    assert ey.max() <= 1.0 and ex.max() <= 1.0 and e.max() <= TOL_DH


def test_beyond_32bit_offsets():
    # 2^16 tokens x 4 streams x C = 16384 bf16: 8 GB per stream tensor, byte offsets pass 2^32
    # at token 2^15; samples on both sides of it and at the end
    B, C = 1 << 16, 16384
    say(f"test: mix B={B} C={C} bf16 (8 GB per stream tensor)")
    H, X, G = workloads.mix_streams_device(B, C, 61, "cuda")
    Y, P, _, it = b4.mix_fwd(H, X, want_iters=True)
    dX, dH = b4.mix_bwd(P, X, G)
    torch.cuda.synchronize()
    assert (it >= 0).all().item()
    idx = np.unique(np.concatenate([np.arange((1 << 15) - 40, (1 << 15) + 40), np.arange(B - 40, B),
                                    np.random.default_rng(5).choice(B, 60, replace=False)]))
    ti = torch.from_numpy(idx).cuda()
    Hs, Xs, Gs = H[ti].float().cpu().numpy(), X[ti].float().cpu().numpy(), G[ti].float().cpu().numpy()
    Yr, Pr = o_fwd(Hs, Xs)
    dXr, dHr = o_bwd(Pr, Xs, Gs)
    assert np.abs(P[ti].cpu().numpy() - Pr).max() <= TOL_P
    ey = np.abs(Y[ti].float().cpu().numpy() - Yr) / mixed_bound(TOL_P, Xs, Yr, True)
    ex = np.abs(dX[ti].float().cpu().numpy() - dXr) / mixed_bound(TOL_P, Gs, dXr, True)
    e = np.abs(dH[ti].cpu().numpy() - dHr).max(axis=(1, 2)) / np.maximum(1.0, np.abs(dHr).max(axis=(1, 2)))
    say(f"  sample of {len(idx)}: Y err/bound={ey.max():.3f} dX err/bound={ex.max():.3f} dH rel={e.max():.2e}")
    assert ey.max() <= 1.0 and ex.max() <= 1.0 and e.max() <= TOL_DH



# The n = 8 kernels take one token per block (a quarter of each row's 16-byte chunks per wave)
# from nc = 256 chunks a row on, one token per wave below: cases on both sides of the switch
# (bf16 C = 2040, 2048, 2056 are nc = 255, 256, 257), ragged last chunks on each wave, and
# fewer tokens than blocks.
CASES8 = [(1, 8, torch.bfloat16, 1.0), (9, 40, torch.float32, 5.0), (300, 520, torch.bfloat16, 5.0),
          (1000, 4096, torch.bfloat16, 20.0), (2049, 1028, torch.float32, 1.0), (64, 0, torch.bfloat16, 5.0),
          (130, 2040, torch.bfloat16, 5.0), (130, 2048, torch.bfloat16, 5.0), (257, 2056, torch.bfloat16, 5.0),
          (517, 1032, torch.float32, 5.0), (3, 4096, torch.bfloat16, 5.0), (700, 1800, torch.float32, 5.0)]


@pytest.mark.parametrize("B,C,dtype,sigma", CASES8,
                         ids=[f"B{b}-C{c}-{str(d)[6:]}-s{s:g}" for b, c, d, s in CASES8])
def test_parity_8_streams(B, C, dtype, sigma):
    say(f"test: 8-stream mix parity B={B} C={C} {dtype} sigma={sigma}")
    H = sigma * np.random.default_rng(B + C + 1).standard_normal((B, 8, 8), dtype=np.float32)
    rng = np.random.default_rng(np.random.SeedSequence([B, C, 88]))
    X = rng.standard_normal((B, 8, C), dtype=np.float32)
    G = rng.standard_normal((B, 8, C), dtype=np.float32)
    if dtype == torch.bfloat16:
        X = workloads.bf16_to_f32(workloads.bf16_bits(X))
        G = workloads.bf16_to_f32(workloads.bf16_bits(G))
    check_case(H, X, G, dtype, f"n=8 B={B} C={C}")


def test_8_streams_autograd_and_workload():
    say("test: 8-stream mix autograd on the mixture workload")
    H, X, G = workloads.mix_streams_device(3000, 256, 62, "cuda", n=8)
    Hr = H.float().requires_grad_()
    Xr = X.clone().requires_grad_()
    Y = b4.mix(Hr, Xr)
    (Y.float() * G.float()).sum().backward()
    Y2, P, _, _ = b4.mix8_fwd(H.float(), X)
    dX, dH = b4.mix8_bwd(P, X, G)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y2) and torch.equal(Hr.grad, dH) and torch.equal(Xr.grad, dX)
    check_case(H.float().cpu().numpy(), X.float().cpu().numpy(), G.float().cpu().numpy(), torch.bfloat16,
               "n=8 mixture")
