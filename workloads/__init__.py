"""Seeded synthetic inputs for the batched 4x4 Birkhoff projection.

This module only draws random numbers and lays them out. It holds none of the
projection's arithmetic, so the HIP path, the CPU oracle, the tests and the
benchmark can all consume what it makes without sharing method code.

Input recipe (the paper's workloads are i.i.d. 4x4 logit matrices, Section 5:
N(0,1), Unif(-1,1), N(0,10^2), Unif(-10,10); its runtime sweep uses N(0,10^2)):

* every batch is split into chunks of ``CHUNK`` matrices; chunk ``c`` of
  workload ``w`` under seed ``s`` draws from
  ``numpy.random.default_rng(SeedSequence([s, w.ident, c]))`` so that any chunk
  can be regenerated on the host alone (sampled oracle checks at full size);
* inside a chunk the draw order is: per-matrix parameters (kinds, scales,
  permutations), then the logits ``H``, then the upstream gradient ``dP``;
* bf16 storage is round-to-nearest-even of the fp32 draw; the oracle sees
  exactly the rounded values, widened back to fp32/fp64.

Arrays are ``[B][4][4]`` row-major float32 (``H``, ``dP``); bf16 arrays are
returned as their raw ``uint16`` bit patterns.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

CHUNK = 1 << 20

# All 24 permutations of (0,1,2,3), in lexicographic order.
PERMS4 = np.array(
    [
        (a, b, c, d)
        for a in range(4)
        for b in range(4)
        for c in range(4)
        for d in range(4)
        if len({a, b, c, d}) == 4
    ],
    dtype=np.int64,
)


@dataclass(frozen=True)
class Workload:
    name: str
    ident: int
    B: int
    kind: str            # "gauss" | "mixture" | "logunif"
    sigma: float = 1.0   # gauss: H = sigma * N(0,1)
    lo: float = 0.1      # logunif: scale log-uniform on [lo, hi]
    hi: float = 50.0
    storage: str = "f32"  # "f32" | "bf16"
    grad: bool = True     # draw an upstream gradient dP
    desc: str = ""


WORKLOADS = {
    w.name: w
    for w in [
        Workload("n01_b4096", 1, 4096, "gauss", sigma=1.0,
                 desc="B=4096 fp32, H ~ N(0,1), dP ~ N(0,1); fwd + bwd"),
        Workload("n01_b2e20_fwd", 2, 1 << 20, "gauss", sigma=1.0, grad=False,
                 desc="B=2^20 fp32, H ~ N(0,1); forward only (P + 8 dual scalars)"),
        Workload("n10_b2e22", 3, 1 << 22, "gauss", sigma=10.0,
                 desc="B=2^22 fp32, H ~ 10 N(0,1), dP ~ N(0,1); fwd + bwd"),
        Workload("mix_bf16_b2e24", 4, 1 << 24, "mixture", storage="bf16",
                 desc="B=2^24 bf16 storage, fp32 compute; half sigma*N(0,1) with "
                      "sigma in {1,5,20}, half 20*Pi + 0.1 N(0,1); kinds shuffled; "
                      "dP ~ N(0,1) bf16; fwd + bwd"),
        Workload("logunif_b2e25", 5, 1 << 25, "logunif", lo=0.1, hi=50.0,
                 desc="B=2^25 fp32, H = a N(0,1), a log-uniform on [0.1, 50] per "
                      "matrix, dP ~ N(0,1); fwd + bwd (+ 20-step Sinkhorn baseline)"),
    ]
}


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); return the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to the fp32 values they encode (exact)."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Chunk:
    H: np.ndarray                 # float32 [n,4,4] (bf16-rounded values if storage == bf16)
    dP: np.ndarray | None         # float32 [n,4,4] or None
    H_bits: np.ndarray | None     # uint16 [n,4,4] when storage == bf16
    dP_bits: np.ndarray | None
    scale: np.ndarray             # float32 [n]: the per-matrix logit scale
    kind: np.ndarray              # int8 [n]: 0 gauss, 1 near-permutation


def _chunk_bounds(w: Workload, B: int, c: int) -> tuple[int, int]:
    lo = c * CHUNK
    return lo, min(B, lo + CHUNK)


def make_chunk(w: Workload, c: int, seed: int = 0, B: int | None = None) -> Chunk:
    """Draw chunk ``c`` of workload ``w`` (matrices [c*CHUNK, min(B, (c+1)*CHUNK)))."""
    B = w.B if B is None else B
    lo, hi = _chunk_bounds(w, B, c)
    n = hi - lo
    rng = np.random.default_rng(np.random.SeedSequence([seed, w.ident, c]))
    kind = np.zeros(n, np.int8)
    # 1) per-matrix parameters
    if w.kind == "gauss":
        scale = np.full(n, w.sigma, np.float32)
        perm = None
    elif w.kind == "mixture":
        kind = (rng.permutation(n) % 2).astype(np.int8)  # exactly half of each, shuffled
        scale = rng.choice(np.array([1.0, 5.0, 20.0], np.float32), size=n)
        perm = rng.integers(0, 24, size=n)
    elif w.kind == "logunif":
        scale = np.exp(rng.uniform(np.log(w.lo), np.log(w.hi), size=n)).astype(np.float32)
        perm = None
    else:
        raise ValueError(w.kind)
    # 2) logits
    z = np.empty((n, 4, 4), np.float32)
    rng.standard_normal(out=z, dtype=np.float32)
    if w.kind == "mixture":
        H = np.where(kind[:, None, None] == 0, scale[:, None, None] * z, np.float32(0.1) * z)
        near = np.nonzero(kind == 1)[0]
        rows = np.arange(4)
        H[near[:, None], rows[None, :], PERMS4[perm[near]]] += np.float32(20.0)
        scale = np.where(kind == 1, np.float32(20.0), scale).astype(np.float32)
    else:
        H = scale[:, None, None] * z
    H = H.astype(np.float32)
    # 3) upstream gradient
    dP = None
    if w.grad:
        dP = np.empty((n, 4, 4), np.float32)
        rng.standard_normal(out=dP, dtype=np.float32)
    H_bits = dP_bits = None
    if w.storage == "bf16":
        H_bits = bf16_bits(H)
        H = bf16_to_f32(H_bits)
        if dP is not None:
            dP_bits = bf16_bits(dP)
            dP = bf16_to_f32(dP_bits)
    return Chunk(H, dP, H_bits, dP_bits, scale, kind)


def n_chunks(w: Workload, B: int | None = None) -> int:
    B = w.B if B is None else B
    return (B + CHUNK - 1) // CHUNK


def generate(name: str, seed: int = 0, B: int | None = None, threads: int = 8) -> Chunk:
    """Draw a whole workload (or its first ``B`` matrices) chunk by chunk.

    Chunks are independent streams, so they are drawn in parallel threads
    (NumPy releases the GIL while filling arrays); the result does not depend
    on ``threads``.
    """
    w = WORKLOADS[name]
    B = w.B if B is None else B
    k = n_chunks(w, B)
    with ThreadPoolExecutor(max(1, min(threads, k))) as ex:
        parts = list(ex.map(lambda c: make_chunk(w, c, seed, B), range(k)))
    if k == 1:
        return parts[0]

    def cat(field):
        xs = [getattr(p, field) for p in parts]
        return None if xs[0] is None else np.concatenate(xs)

    return Chunk(*(cat(f) for f in ("H", "dP", "H_bits", "dP_bits", "scale", "kind")))


def gauss(B: int, sigma: float, seed: int, grad: bool = True) -> tuple[np.ndarray, np.ndarray | None]:
    """Small ad-hoc batch: H = sigma * N(0,1) and dP ~ N(0,1) (tests and edge cases)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 1000, int(round(sigma * 1000))]))
    H = (np.float32(sigma) * rng.standard_normal((B, 4, 4), dtype=np.float32)).astype(np.float32)
    dP = rng.standard_normal((B, 4, 4), dtype=np.float32) if grad else None
    return H, dP


def near_permutation(B: int, gap: float, noise: float, seed: int) -> tuple[np.ndarray, np.ndarray]:
    """H = gap * Pi + noise * N(0,1) with Pi uniform over the 24 permutations."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 2000]))
    perm = rng.integers(0, 24, size=B)
    H = (np.float32(noise) * rng.standard_normal((B, 4, 4), dtype=np.float32)).astype(np.float32)
    H[np.arange(B)[:, None], np.arange(4)[None, :], PERMS4[perm]] += np.float32(gap)
    dP = rng.standard_normal((B, 4, 4), dtype=np.float32)
    return H, dP


# ---------------------------------------------------------------------------
# Larger-problem workloads drawn on the GPU with torch's seeded generator (2^28 values take
# a while in NumPy); any sample of them is copied back for the oracle.
# ---------------------------------------------------------------------------

def n8_mix_device(B: int, seed: int, dev):
    """8x8 mixture: half H = sigma * N(0,1) with sigma drawn from {1, 5, 20}, half
    H = 20 Pi + 0.1 N(0,1) for a uniformly random permutation Pi of 8 (kinds shuffled),
    dP ~ N(0,1); both stored as bf16. Returns (H, dP) on ``dev``."""
    import torch
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    Z = torch.randn(B, 8, 8, device=dev, generator=g)
    kind = torch.randint(0, 2, (B,), device=dev, generator=g)
    sig = torch.tensor([1.0, 5.0, 20.0], device=dev)[torch.randint(0, 3, (B,), device=dev, generator=g)]
    perm = torch.argsort(torch.rand(B, 8, device=dev, generator=g), dim=1)
    Pi = torch.zeros(B, 8, 8, device=dev).scatter_(2, perm[:, :, None], 1.0)
    H = torch.where(kind[:, None, None] == 0, sig[:, None, None] * Z, 20.0 * Pi + 0.1 * Z)
    G = torch.randn(B, 8, 8, device=dev, generator=g)
    return H.to(torch.bfloat16).contiguous(), G.to(torch.bfloat16).contiguous()


def ot_device(B: int, seed: int, dev, n: int = 4):
    """n x n entropic-OT problems: cost M = 2 N(0,1), marginals a, b ~ U(0.2, 2) with b
    rescaled (in fp64) to the sum of a, upstream gradient dT ~ N(0,1); fp32. Returns
    (M, a, b, dT) on ``dev``."""
    import torch
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    M = 2.0 * torch.randn(B, n, n, device=dev, generator=g)
    a = 0.2 + 1.8 * torch.rand(B, n, device=dev, generator=g)
    b = 0.2 + 1.8 * torch.rand(B, n, device=dev, generator=g)
    b = (b.double() * (a.double().sum(1) / b.double().sum(1))[:, None]).float()
    G = torch.randn(B, n, n, device=dev, generator=g)
    return M.contiguous(), a.contiguous(), b.contiguous(), G.contiguous()


def mix_streams_device(B: int, C: int, seed: int, dev, n: int = 4):
    """Residual mixing of the mHC layer: per token, n x n logits H from the headline mixture
    (half sigma * N(0,1) with sigma drawn from {1, 5, 20}, half 20 Pi + 0.1 N(0,1) for a
    random permutation Pi, kinds shuffled) and n streams of C channels X ~ N(0,1), with
    upstream gradient dY ~ N(0,1) of the same shape; all stored as bf16. Returns
    (H [B,n,n], X [B,n,C], dY [B,n,C]) on ``dev``."""
    import torch
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    Z = torch.randn(B, n, n, device=dev, generator=g)
    kind = torch.randint(0, 2, (B,), device=dev, generator=g)
    sig = torch.tensor([1.0, 5.0, 20.0], device=dev)[torch.randint(0, 3, (B,), device=dev, generator=g)]
    perm = torch.argsort(torch.rand(B, n, device=dev, generator=g), dim=1)
    Pi = torch.zeros(B, n, n, device=dev).scatter_(2, perm[:, :, None], 1.0)
    H = torch.where(kind[:, None, None] == 0, sig[:, None, None] * Z, 20.0 * Pi + 0.1 * Z)
    X = torch.randn(B, n, C, device=dev, generator=g).to(torch.bfloat16)
    G = torch.randn(B, n, C, device=dev, generator=g).to(torch.bfloat16)
    return H.to(torch.bfloat16).contiguous(), X.contiguous(), G.contiguous()


def uniform(B: int, half_width: float, seed: int, grad: bool = True) -> tuple[np.ndarray, np.ndarray | None]:
    """Small ad-hoc batch: H ~ Unif(-half_width, half_width) and dP ~ N(0,1)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 3000, int(round(half_width * 1000))]))
    H = rng.uniform(-half_width, half_width, size=(B, 4, 4)).astype(np.float32)
    dP = rng.standard_normal((B, 4, 4), dtype=np.float32) if grad else None
    return H, dP
