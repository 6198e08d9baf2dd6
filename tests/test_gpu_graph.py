"""Every entry point captured in a HIP graph (torch.cuda.CUDAGraph) and replayed.

The library only launches kernels on the caller's stream: no allocation, synchronisation or
memset, and no device state that outlives a launch, so a captured call must give the same
bits as the eager call on the same inputs. Each case captures once, then for several input
sets copies the set into the captured input buffers, runs the eager call on the set (the
program's own work between replays), replays the graph twice and compares every output of
both replays bitwise with the eager result.
"""
import pytest
import torch

import paper_2606_07574_amd as b4
import workloads
from tests._gpu import say, to_dev

pytestmark = pytest.mark.gpu

N_SETS = 3


def graph_roundtrip(fn, sets, label):
    static = [t.clone() for t in sets[0]]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn(*static)                      # first call (per-device set-up) outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = [o for o in fn(*static) if o is not None]
    torch.cuda.synchronize()
    for k, inp in enumerate(sets):
        for d, src in zip(static, inp):
            d.copy_(src)
        ref = [o for o in fn(*inp) if o is not None]
        torch.cuda.synchronize()
        for rep in range(2):
            for o in outs:          # poison the outputs so a replay that writes nothing fails
                o.fill_(float("nan") if o.is_floating_point() else -7)
            g.replay()
            torch.cuda.synchronize()
            for i, (o, r) in enumerate(zip(outs, ref)):
                assert torch.equal(o, r), f"{label}: set {k}, replay {rep}, output {i} differs from eager"
        say(f"  [{label}] set {k}: both replays equal the eager call")


def gauss_sets(B, sigma, dtype=torch.float32, seed=0):
    sets = []
    for k in range(N_SETS):
        H, dP = workloads.gauss(B, sigma, seed=seed + k)
        sets.append([to_dev(H, dtype), to_dev(dP, dtype)])
    return sets


@pytest.mark.parametrize("variant,B,dtype", [(b4.THROUGHPUT, 20011, torch.float32),
                                             (b4.LATENCY, 4096, torch.float32),
                                             (b4.THROUGHPUT, 4097, torch.bfloat16),
                                             (b4.LATENCY, 1000, torch.bfloat16)],
                         ids=["throughput-f32", "latency-f32", "throughput-bf16", "latency-bf16"])
def test_graph_fwd_bwd(variant, B, dtype):
    say(f"test: graph capture fwd + bwd, variant {variant}, B={B}, {dtype}")

    def fn(H, dP):
        P, dual, it = b4.fwd(H, 1e-6, 64, want_dual=True, want_iters=True, variant=variant)
        return P, dual, it, b4.bwd(P, dP)

    graph_roundtrip(fn, gauss_sets(B, 5.0, dtype, seed=11), f"4x4 {variant}")


def test_graph_saved_hessian():
    say("test: graph capture of the saved-Hessian pair")

    def fn(H, dP):
        P, dual, hess, it = b4.fwd_hess(H, 1e-6, 64, want_dual=True, want_iters=True)
        return P, dual, hess, it, b4.bwd_hess(P, hess, dP)

    graph_roundtrip(fn, gauss_sets(5003, 5.0, seed=21), "saved Hessian")


def test_graph_sinkhorn():
    say("test: graph capture of the Sinkhorn-Knopp baseline")

    def fn(H, dP):
        return b4.sk_fwd(H, 20), b4.sk_bwd(H, dP, 20)

    graph_roundtrip(fn, gauss_sets(4099, 5.0, seed=31), "SK-20")


def test_graph_n8():
    say("test: graph capture of the 8x8 pair")
    sets = []
    for k in range(N_SETS):
        g = torch.Generator(device="cuda").manual_seed(40 + k)
        H = 5.0 * torch.randn(3001, 8, 8, device="cuda", generator=g)
        dP = torch.randn(3001, 8, 8, device="cuda", generator=g)
        sets.append([H, dP])

    def fn(H, dP):
        P, dual, it = b4.fwd8(H, 1e-6, 64, want_dual=True, want_iters=True)
        return P, dual, it, b4.bwd8(P, dP)

    graph_roundtrip(fn, sets, "8x8")


@pytest.mark.parametrize("n", [4, 8])
def test_graph_ot(n):
    say(f"test: graph capture of the {n}x{n} OT pair")
    sets = []
    for k in range(N_SETS):
        M, a, b, G = workloads.ot_device(2999, 50 + k, "cuda", n)
        sets.append([M, a, b, G])
    fwd, bwd = (b4.ot_fwd, b4.ot_bwd) if n == 4 else (b4.ot8_fwd, b4.ot8_bwd)

    def fn(M, a, b, G):
        T, dual, it = fwd(M, a, b, 0.5, 1e-6, 64, want_dual=True, want_iters=True)
        return T, dual, it, bwd(T, a, G, 0.5)

    graph_roundtrip(fn, sets, f"OT {n}x{n}")


def test_graph_many_launches():
    # a graph of 16 fwd + bwd pairs on independent small batches (the launch-bound case):
    # every pair's outputs equal the eager call's
    say("test: graph of 16 small fwd + bwd pairs")
    sets = gauss_sets(512 * 16, 20.0, seed=61)

    def fn(H, dP):
        outs = []
        for j in range(16):
            h, d = H[512 * j:512 * (j + 1)], dP[512 * j:512 * (j + 1)]
            P, _, it = b4.fwd(h, 1e-6, 64, want_dual=False, want_iters=True)
            outs += [P, it, b4.bwd(P, d)]
        return outs

    graph_roundtrip(fn, sets, "16 pairs")


# C = 2048 bf16 channels (256 chunks a row) puts the 8-stream kernels on one token per block
@pytest.mark.parametrize("n,C", [(4, 264), (8, 264), (8, 2048)])
def test_graph_mix(n, C):
    say(f"test: graph capture of the residual-mixing pair, {n} streams, C={C}")
    sets = [list(workloads.mix_streams_device(3001 if C < 1024 else 700, C, 70 + k, "cuda", n))
            for k in range(N_SETS)]
    mfwd, mbwd = (b4.mix_fwd, b4.mix_bwd) if n == 4 else (b4.mix8_fwd, b4.mix8_bwd)

    def fn(H, X, G):
        Y, P, _, it = mfwd(H, X, 1e-6, 64, want_iters=True)
        dX, dH = mbwd(P, X, G)
        return Y, P, it, dX, dH

    graph_roundtrip(fn, sets, "mix")
