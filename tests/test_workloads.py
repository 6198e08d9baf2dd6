"""The seeded input generators: determinism, chunk independence, bf16 rounding."""
import numpy as np
import torch

import workloads


def test_bf16_round_to_nearest_even_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    x[:4] = [1.0 + 2**-8, 1.0 + 3 * 2**-8, -(1.0 + 2**-8), 0.0]  # ties
    bits = workloads.bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (bits == ref).all()
    back = workloads.bf16_to_f32(bits)
    assert (back == torch.from_numpy(x).to(torch.bfloat16).float().numpy()).all()


def test_chunks_are_reproducible_and_independent():
    w = workloads.WORKLOADS["logunif_b2e25"]
    B = 2 * workloads.CHUNK + 1000
    full = workloads.generate(w.name, B=B, threads=3)
    c1 = workloads.make_chunk(w, 1, B=B)
    assert np.array_equal(full.H[workloads.CHUNK:2 * workloads.CHUNK], c1.H)
    assert np.array_equal(full.dP[workloads.CHUNK:2 * workloads.CHUNK], c1.dP)
    last = workloads.make_chunk(w, 2, B=B)
    assert last.H.shape == (1000, 4, 4)
    assert np.array_equal(full.H[-1000:], last.H)
    assert 0.1 <= full.scale.min() and full.scale.max() <= 50.0


def test_mixture_recipe():
    w = workloads.WORKLOADS["mix_bf16_b2e24"]
    ch = workloads.make_chunk(w, 0, B=40000)
    assert ch.H_bits.dtype == np.uint16 and ch.dP_bits is not None
    assert ch.kind.sum() == 20000  # exactly half near-permutations
    near = ch.kind == 1
    big = (ch.H[near] > 10).sum(axis=2)
    assert (big == 1).all() and ((ch.H[near] > 10).sum(axis=1) == 1).all()
    sig = set(np.unique(ch.scale[~near]).tolist())
    assert sig == {1.0, 5.0, 20.0}
    # kinds are interleaved, not split in halves
    assert 0.3 < ch.kind[:64].mean() < 0.7 or 0.3 < ch.kind[64:128].mean() < 0.7


def test_config_table():
    B = {k: w.B for k, w in workloads.WORKLOADS.items()}
    assert B == {"n01_b4096": 4096, "n01_b2e20_fwd": 1 << 20, "n10_b2e22": 1 << 22,
                 "mix_bf16_b2e24": 1 << 24, "logunif_b2e25": 1 << 25}


def test_device_generators_on_cpu():
    import torch
    H, G = workloads.n8_mix_device(300, 8, "cpu")
    assert H.shape == (300, 8, 8) and G.shape == (300, 8, 8) and H.dtype == torch.bfloat16
    H2, _ = workloads.n8_mix_device(300, 8, "cpu")
    assert torch.equal(H, H2)
    # about half are near-permutations: one entry per row within 0.6 of 20, at distinct
    # columns, every other entry within 0.6 of 0
    Hf = H.float()
    near20 = (Hf - 20).abs() < 0.6
    rest_small = torch.where(near20, torch.zeros_like(Hf), Hf).abs().amax(dim=(1, 2)) < 0.6
    is_perm = (near20.sum(2) == 1).all(1) & (near20.sum(1) == 1).all(1) & rest_small
    assert 0.35 < is_perm.float().mean().item() < 0.65
    M, a, b, dT = workloads.ot_device(500, 4, "cpu")
    assert M.shape == (500, 4, 4) and a.shape == (500, 4) and b.shape == (500, 4) and dT.shape == (500, 4, 4)
    assert (a >= 0.2).all() and (a <= 2.0).all() and (b > 0).all()
    assert (a.double().sum(1) - b.double().sum(1)).abs().max() < 1e-5


def test_mix_streams_generator_on_cpu():
    import torch
    H, X, G = workloads.mix_streams_device(400, 24, 60, "cpu")
    assert H.shape == (400, 4, 4) and X.shape == (400, 4, 24) and G.shape == (400, 4, 24)
    assert H.dtype == X.dtype == G.dtype == torch.bfloat16
    H2, X2, _ = workloads.mix_streams_device(400, 24, 60, "cpu")
    assert torch.equal(H, H2) and torch.equal(X, X2)
    Hf = H.float()
    near20 = (Hf - 20).abs() < 0.6
    rest_small = torch.where(near20, torch.zeros_like(Hf), Hf).abs().amax(dim=(1, 2)) < 0.6
    is_perm = (near20.sum(2) == 1).all(1) & (near20.sum(1) == 1).all(1) & rest_small
    assert 0.35 < is_perm.float().mean().item() < 0.65
    assert abs(X.float().std().item() - 1.0) < 0.05
