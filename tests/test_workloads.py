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
