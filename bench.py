#!/usr/bin/env python3
"""Throughput of the batched 4x4 Birkhoff projection (forward + backward) on one MI355X.

One step = one pass of the whole path over the batch: the Newton forward kernel
(H -> P, dual) followed by the implicit-differentiation backward kernel
(P, dP -> dH), both launched through the C ABI on torch's current stream. Inputs
are synthetic (workloads/), generated on the host and resident in HBM before the
timed region. Prints ONE JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload mix_bf16_b2e24]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "4×4 Birkhoff projections/sec fwd+bwd at B=2^24 (fp32); % HBM peak; max marginal err"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
# VALU issue peak without packed fp32: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz lane-instructions/s
VALU_PEAK_T = 256 * 4 * 16 * 2.4e9 / 1e12
SRC = os.path.join(ROOT, "paper_2606_07574_amd", "csrc", "birkhoff4.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def in_bytes(dtype_is_bf16: bool) -> int:
    return 32 if dtype_is_bf16 else 64


def valu_from_profiles(workload: str, kernel: str, kind: str = "valu"):
    """VALU lane-instructions per launch counted by rocprofv3 (SQ_INSTS_VALU x 64) for the
    current kernel source (profiles/<kind>_<workload>.md), else None."""
    path = os.path.join(ROOT, "profiles", f"{kind}_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    if not m or m.group(1) != hashlib.sha256(open(SRC, "rb").read()).hexdigest():
        return None
    mm = re.search(rf"{kernel}_valu_lane_instr_per_launch:\s*([0-9.eE+]+)", text)
    return float(mm.group(1)) if mm else None


def profile_figure(fname: str, key: str):
    """A `key: value` figure of profiles/<fname>, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", fname)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"source_sha256[^:]*:\s*([0-9a-f]{64})", text)
    if not m or m.group(1) != hashlib.sha256(open(SRC, "rb").read()).hexdigest():
        return None
    mm = re.search(rf"{key}:\s*([0-9.eE+]+)", text)
    return float(mm.group(1)) if mm else None


def traffic_from_profiles(workload: str):
    """HBM bytes per launch measured by rocprofv3 counters, if they were taken on
    the current kernel source (profiles/traffic_<workload>.md)."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    src = hashlib.sha256(open(SRC, "rb").read()).hexdigest()
    if not m or m.group(1) != src:
        return None
    out = {}
    for k in ("newton_fwd", "implicit_bwd"):
        mm = re.search(rf"{k}_hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
        if mm:
            out[k] = float(mm.group(1))
    return out or None


# The paper's accuracy tables (Sec. 5, Tables 1-2): L1 marginal error ||T1 - 1||_1 + ||T^T 1 - 1||_1
# over 10,000 matrices, mean / std / median / max; measured on an NVIDIA RTX 6000 Ada, precision not
# stated, Newton at tol 1e-6 and at most 20 iterations, Sinkhorn-Knopp ("Vanilla") 20 iterations.
PAPER_TABLES = {
    "N(0,1)": {"newton": [0.654e-6, 0.385e-6, 0.527e-6, 2.503e-6], "sk20": [8.336e-6, 20.01e-6, 7.793e-6, 1381e-6]},
    "Unif(-1,1)": {"newton": [0.593e-6, 0.352e-6, 0.477e-6, 2.325e-6], "sk20": [7.790e-6, 0.141e-6, 7.793e-6, 8.330e-6]},
    "N(0,10^2)": {"newton": [1.594e-3, 4.428e-3, 0.0009e-3, 91.3e-3], "sk20": [72.54e-3, 61.12e-3, 65.13e-3, 832.6e-3]},
    "Unif(-10,10)": {"newton": [0.159e-3, 1.479e-3, 0.0006e-3, 46.57e-3], "sk20": [40.02e-3, 37.16e-3, 32.93e-3, 234.0e-3]},
}
PAPER_CAP = 20  # the paper's iteration cap (Sec. 5)


def step_stats(itn: np.ndarray) -> dict:
    """Newton trial evaluations per matrix; frac_over_20: the share that the paper's cap of 20
    iterations would leave unconverged (this library counts every trial evaluation)."""
    conv = itn[itn >= 0]
    n64 = (len(itn) // 64) * 64
    wave_max = np.clip(itn[:n64], 0, None).reshape(-1, 64).max(axis=1).mean() if n64 else float("nan")
    return {"mean": round(float(conv.mean()), 3) if len(conv) else None,
            "p50": int(np.percentile(conv, 50)) if len(conv) else None,
            "p99": int(np.percentile(conv, 99)) if len(conv) else None,
            "max": int(conv.max()) if len(conv) else None,
            "mean_of_wave_max": round(float(wave_max), 3),
            "not_converged": int((itn == -1).sum()), "non_finite": int((itn == -2).sum()),
            "frac_over_20": float(((itn > PAPER_CAP) | (itn == -1)).mean()),
            "hist": np.bincount(np.clip(conv, 0, 40), minlength=41).tolist()}


def l1_stats(P) -> tuple:
    """Per-matrix max marginal error and the paper's L1 error, in fp64 on the device."""
    P64 = P.double()
    r, c = P64.sum(-1) - 1, P64.sum(-2) - 1
    marg = torch_max(r.abs().amax(-1), c.abs().amax(-1))
    l1 = r.abs().sum(-1) + c.abs().sum(-1)
    return marg, l1


def torch_max(a, b):
    import torch
    return torch.maximum(a, b)


def measure(name, args, dev, stream, *, storage=None, steps=None, warmup=None, extras=True, sk=False,
            buckets=False, autograd=False, hess=False):
    """Time K steps of the whole path (forward, and backward when the workload has dP) on one
    workload through the C ABI, inputs resident in HBM; per-kernel HIP-event times on the
    launch stream. storage="f32" stores a bf16 workload's (bf16-rounded) values as fp32."""
    import torch

    import paper_2606_07574_amd as b4
    import workloads
    w = workloads.WORKLOADS[name]
    B = w.B
    t0 = time.time()
    ch = workloads.generate(w.name, threads=16)
    log(f"generated {w.name} B={B} in {time.time() - t0:.1f}s")
    bf16 = w.storage == "bf16" and storage != "f32"

    def dev_input(x32, bits):
        if bf16 and bits is not None:
            return torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(x32).to(dev)

    # working set per buffer set; rotate sets so the 256 MB last-level cache cannot hold it
    set_bytes = B * (in_bytes(bf16) + 64 + 32 + ((in_bytes(bf16) + 64) if w.grad else 0))
    n_sets = max(1, min(8, math.ceil((768 << 20) / set_bytes)))
    sets = []
    H0 = dev_input(ch.H, ch.H_bits)
    G0 = dev_input(ch.dP, ch.dP_bits) if w.grad else None
    for s in range(n_sets):
        Hs = H0 if s == 0 else H0.clone()
        Gs = (G0 if s == 0 else G0.clone()) if w.grad else None
        sets.append(dict(H=Hs, G=Gs, P=torch.empty(B, 4, 4, device=dev),
                         dual=torch.empty(B, 8, device=dev),
                         dH=torch.empty(B, 4, 4, device=dev) if w.grad else None))
    torch.cuda.synchronize()
    lib = b4.lib()
    sptr = stream.cuda_stream
    hcode = b4.BF16 if bf16 else b4.F32
    K = args.steps if steps is None else steps
    W = args.warmup if warmup is None else warmup
    ev_start = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
    ev_mid = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
    ev_end = [torch.cuda.Event(enable_timing=True) for _ in range(K)]

    def step(k, timed):
        st = sets[k % n_sets]
        if timed:
            ev_start[k].record(stream)
        rc = lib.birkhoff4_fwd_ex(st["H"].data_ptr(), hcode, st["P"].data_ptr(), st["dual"].data_ptr(),
                                  None, B, args.tol, args.max_iter, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())
        if timed:
            ev_mid[k].record(stream)
        if w.grad:
            rc = lib.birkhoff4_bwd_ex(st["P"].data_ptr(), st["G"].data_ptr(), hcode,
                                      st["dH"].data_ptr(), B, sptr)
            if rc:
                raise RuntimeError(lib.birkhoff4_strerror(rc).decode())
        if timed:
            ev_end[k].record(stream)

    for k in range(W):
        step(k, False)
    torch.cuda.synchronize()
    log(f"{w.name}: warmup done ({W} steps); timing {K} steps")
    t_start = time.perf_counter()
    for k in range(K):
        step(k, True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    fwd_ms = float(np.mean([ev_start[k].elapsed_time(ev_mid[k]) for k in range(K)]))
    bwd_ms = float(np.mean([ev_mid[k].elapsed_time(ev_end[k]) for k in range(K)])) if w.grad else 0.0
    ms_per_step = wall * 1e3 / K
    log(f"{w.name}{' (fp32 storage)' if storage == 'f32' else ''} timed: {ms_per_step:.3f} ms/step  "
        f"fwd {fwd_ms:.3f} ms  bwd {bwd_ms:.3f} ms")
    fwd_bytes = B * (in_bytes(bf16) + 64 + 32)
    bwd_bytes = B * (64 + in_bytes(bf16) + 64)
    kernels = {"newton_fwd": {"avg_ms": fwd_ms, "alg_bytes_per_launch": fwd_bytes,
                              "achieved_GBs": fwd_bytes / (fwd_ms * 1e-3) / 1e9,
                              "proj_per_s": B / (fwd_ms * 1e-3)}}
    if w.grad:
        kernels["implicit_bwd"] = {"avg_ms": bwd_ms, "alg_bytes_per_launch": bwd_bytes,
                                   "achieved_GBs": bwd_bytes / (bwd_ms * 1e-3) / 1e9,
                                   "proj_per_s": B / (bwd_ms * 1e-3)}
    path_bytes = fwd_bytes + (bwd_bytes if w.grad else 0)
    res = {"workload": w.name + ("_f32_storage" if storage == "f32" else ""), "B": B,
           "storage": "bf16" if bf16 else "f32", "passes": "fwd+bwd" if w.grad else "fwd",
           "desc": w.desc + (" -- stored as fp32 (the same bf16-rounded values)" if storage == "f32" else ""),
           "steps": K, "buffer_sets": n_sets, "ms_per_step": round(ms_per_step, 4),
           "value": round(B * K / wall, 1), "unit": "proj/s",
           "alg_bytes_per_projection": path_bytes // B,
           "path_hbm_frac": round(path_bytes * K / wall / 1e9 / HBM_PEAK_GBS, 4),
           "kernels": {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                       for k, v in kernels.items()}}
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"])
    ach = kernels[dom]["achieved_GBs"]
    res["roofline"] = {"bound": "hbm", "kernel": dom, "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                       "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4)}
    res["_wall"], res["_fwd_ms"], res["_lib"], res["_hcode"] = wall, fwd_ms, lib, hcode
    if extras:
        # outside the timed region: Newton step histogram, marginal errors
        st = sets[0]
        P, dual, it = b4.fwd(st["H"], args.tol, args.max_iter, want_dual=True, want_iters=True)
        torch.cuda.synchronize()
        itn = it.cpu().numpy()
        marg, l1 = l1_stats(P)
        res["newton_steps"] = step_stats(itn)
        res["max_marginal_err"] = float(marg.max().item())
        res["marginal_err_L1"] = {"mean": float(l1.mean().item()), "median": float(l1.median().item()),
                                  "max": float(l1.max().item())}
        log(f"{w.name}: newton steps {res['newton_steps']}; max marginal err {res['max_marginal_err']:.3e}")
        sk_marg = None
        if sk:
            n_sk = 20
            for _ in range(2):
                b4.sk_fwd(st["H"], n_sk)
                if w.grad:
                    b4.sk_bwd(st["H"], st["G"], n_sk)
            torch.cuda.synchronize()
            e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            ks = max(3, K // 4)
            f_ms = b_ms = 0.0
            for k in range(ks):
                e0.record(stream)
                Psk = b4.sk_fwd(sets[k % n_sets]["H"], n_sk)
                e1.record(stream)
                if w.grad:
                    b4.sk_bwd(sets[k % n_sets]["H"], sets[k % n_sets]["G"], n_sk)
                e2.record(stream)
                torch.cuda.synchronize()
                f_ms += e0.elapsed_time(e1)
                b_ms += e1.elapsed_time(e2) if w.grad else 0.0
            f_ms /= ks
            b_ms /= ks
            smarg, sl1 = l1_stats(Psk)
            res["sk20_baseline"] = {
                "value": round(B / ((f_ms + b_ms) * 1e-3), 1), "unit": "proj/s",
                "fwd_ms": round(f_ms, 4), "bwd_ms": round(b_ms, 4),
                "max_marginal_err": float(smarg.max().item()),
                "marginal_err_L1": {"mean": float(sl1.mean().item()), "median": float(sl1.median().item()),
                                    "max": float(sl1.max().item())},
            }
            log(f"{w.name}: sk20 {res['sk20_baseline']}")
            sk_marg = smarg.cpu().numpy()
            del Psk
        if buckets:
            res["buckets"] = bucket_report(w, ch, itn, marg.cpu().numpy(), sk_marg)
        del P, dual, it, marg, l1
        if autograd and w.grad:
            res["autograd_step"] = bench_autograd_step(args, lib, sets, n_sets, B, hcode, bf16, stream,
                                                       in_bytes(bf16))
            log(f"autograd step (no dual): {res['autograd_step']}")
        if hess and w.grad:
            res["saved_hessian"] = bench_saved_hessian(args, lib, sets, n_sets, B, hcode, bf16, stream,
                                                       in_bytes(bf16), ms_per_step)
            log(f"saved hessian: {res['saved_hessian']}")
    res["_ch"] = ch
    del sets, H0, G0
    return res


def public(res: dict) -> dict:
    return {k: v for k, v in res.items() if not k.startswith("_")}


def bench_b4096(args, dev) -> dict:
    """n01_b4096 (B = 4096 N(0,1) fp32 matrices): launch-bound, reported in microseconds per
    fwd + bwd call pair, eager and replayed from a HIP graph, plus each kernel's event time."""
    import torch

    import paper_2606_07574_amd as b4
    import workloads
    ch = workloads.make_chunk(workloads.WORKLOADS["n01_b4096"], 0)
    row = bench_small_batch(dev, sizes=(4096,), inputs={4096: (ch.H, ch.dP)})[0]
    H = torch.from_numpy(ch.H).to(dev)
    P, dual, it = b4.fwd(H, args.tol, args.max_iter, want_dual=True, want_iters=True)
    torch.cuda.synchronize()
    marg, l1 = l1_stats(P)
    return {"workload": "n01_b4096", "B": 4096, "desc": workloads.WORKLOADS["n01_b4096"].desc,
            "unit": "us per fwd+bwd call pair", "eager_us_per_pair": row["eager_us_per_pair"],
            "graph_us_per_pair": row["graph_us_per_pair"], "fwd_event_us": row["fwd_event_us"],
            "bwd_event_us": row["bwd_event_us"], "graph_proj_per_s": row["graph_proj_per_s"],
            "newton_steps": step_stats(it.cpu().numpy()), "max_marginal_err": float(marg.max().item())}


# The paper's runtime table (Sec. 5, Table 3): median run times on N(0,10^2) logits, normalised
# so that its own CUDA solver takes 1, on an NVIDIA RTX 6000 Ada. Columns: an unfused PyTorch
# Sinkhorn (Vanilla), Triton Sinkhorn, mHC.cu, TileLang examples (TLE), TileKernels (TK) and
# its TileLang Newton solver (Proj-TL); rows by batch size (1K = 1024).
PAPER_RUNTIME = {
    "columns": ["Vanilla", "Triton", "mHC.cu", "TLE", "TK", "Proj-TL"],
    "fwd": {512: [49.778, 9.449, 2.908, 3.092, 2.862, 2.925], 2048: [49.974, 18.811, 2.977, 3.106, 2.867, 2.946],
            8192: [49.289, 89.064, 4.307, 3.644, 2.830, 2.859], 32768: [22.879, 197.626, 2.354, 5.399, 2.262, 1.377],
            131072: [12.419, 337.584, 1.674, 6.887, 3.001, 1.235]},
    "fwd_bwd": {512: [126.380, 9.754, 3.548, 3.066, 3.058, 3.071], 2048: [125.481, 12.835, 3.595, 3.046, 3.034, 3.048],
                8192: [124.970, 56.654, 4.367, 3.076, 8.498, 3.048],
                32768: [103.678, 213.621, 7.809, 4.984, 22.028, 2.497],
                131072: [51.518, 376.858, 22.310, 6.329, 28.345, 1.208]},
}


def bench_runtime_table(args, dev, stream, reps: int = 51) -> dict:
    """The paper's runtime sweep on this hardware: N(0,10^2) logits at its five batch sizes,
    median over `reps` calls of the event-timed forward and forward + backward, for the Newton
    path (no dual, default kernel variant) and for this library's fused 20-step Sinkhorn-Knopp
    pair, with SK-20 / Newton ratios beside the paper's normalised columns (context only: other
    hardware, other implementations)."""
    import torch

    import paper_2606_07574_amd as b4
    import workloads
    lib = b4.lib()
    sptr = stream.cuda_stream
    F32 = b4.F32
    rows = []
    for B in (512, 2048, 8192, 32768, 131072):
        H32, G32 = workloads.gauss(B, 10.0, seed=900 + B.bit_length())
        H, G = torch.from_numpy(H32).to(dev), torch.from_numpy(G32).to(dev)
        P, dH, Psk, dHs = (torch.empty_like(H) for _ in range(4))

        def newton_fwd():
            rc = lib.birkhoff4_fwd_ex2(H.data_ptr(), F32, P.data_ptr(), None, None, B, args.tol, args.max_iter,
                                       b4.AUTO, sptr)
            if rc:
                raise RuntimeError(lib.birkhoff4_strerror(rc).decode())

        def newton_bwd():
            rc = lib.birkhoff4_bwd_ex(P.data_ptr(), G.data_ptr(), F32, dH.data_ptr(), B, sptr)
            if rc:
                raise RuntimeError(lib.birkhoff4_strerror(rc).decode())

        def sk_fwd():
            rc = lib.birkhoff4_sk_fwd(H.data_ptr(), F32, Psk.data_ptr(), B, PAPER_CAP, sptr)
            if rc:
                raise RuntimeError(lib.birkhoff4_strerror(rc).decode())

        def sk_bwd():
            rc = lib.birkhoff4_sk_bwd(H.data_ptr(), F32, G.data_ptr(), F32, dHs.data_ptr(), B, PAPER_CAP, sptr)
            if rc:
                raise RuntimeError(lib.birkhoff4_strerror(rc).decode())

        def median_us(calls):
            ts = []
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            for r in range(reps + 3):
                torch.cuda.synchronize()
                e0.record(stream)
                for c in calls:
                    c()
                e1.record(stream)
                torch.cuda.synchronize()
                if r >= 3:
                    ts.append(e0.elapsed_time(e1) * 1e3)
            return float(np.median(ts))

        nf, nfb = median_us([newton_fwd]), median_us([newton_fwd, newton_bwd])
        sf, sfb = median_us([sk_fwd]), median_us([sk_fwd, sk_bwd])
        row = {"B": B, "newton_fwd_us": round(nf, 2), "newton_fwd_bwd_us": round(nfb, 2), "sk20_fwd_us": round(sf, 2),
               "sk20_fwd_bwd_us": round(sfb, 2), "sk20_over_newton_fwd": round(sf / nf, 3),
               "sk20_over_newton_fwd_bwd": round(sfb / nfb, 3),
               "paper_fwd": dict(zip(PAPER_RUNTIME["columns"], PAPER_RUNTIME["fwd"][B])),
               "paper_fwd_bwd": dict(zip(PAPER_RUNTIME["columns"], PAPER_RUNTIME["fwd_bwd"][B]))}
        log(f"runtime table: {row}")
        rows.append(row)
        del H, G, P, dH, Psk, dHs
    return {"logits": "N(0,10^2), fp32", "timing": f"median over {reps} event-timed calls, synchronised between calls",
            "newton": f"default kernel variant (four lanes per problem up to B = 32768), no dual, tol {args.tol}, "
                      f"max_iter {args.max_iter}",
            "sk20": "this library's fused 20-step Sinkhorn-Knopp forward and exact reverse-mode backward",
            "paper": "Sec. 5 Table 3, median times normalised to the paper's CUDA solver (= 1), NVIDIA RTX 6000 Ada",
            "rows": rows}


def bench_accuracy(args, dev) -> dict:
    """The paper's accuracy tables on this hardware: 10,000 matrices from each of its four input
    families, L1 marginal error of the Newton forward and of the 20-step Sinkhorn-Knopp baseline
    (mean / std / median / max), beside the paper's own figures (RTX 6000 Ada)."""
    import torch

    import paper_2606_07574_amd as b4
    import workloads
    fams = {"N(0,1)": workloads.gauss(10000, 1.0, seed=101, grad=False)[0],
            "Unif(-1,1)": workloads.uniform(10000, 1.0, seed=102, grad=False)[0],
            "N(0,10^2)": workloads.gauss(10000, 10.0, seed=103, grad=False)[0],
            "Unif(-10,10)": workloads.uniform(10000, 10.0, seed=104, grad=False)[0]}
    out = {"n": 10000, "measure": "L1 marginal error ||P1-1||_1 + ||P^T1-1||_1 (fp64 sums of the fp32 output)",
           "order": ["mean", "std", "median", "max"], "tol": args.tol, "max_iter": args.max_iter,
           "paper_hardware": "NVIDIA RTX 6000 Ada (paper, Sec. 5; precision not stated)", "families": {}}
    for name, H32 in fams.items():
        H = torch.from_numpy(H32).to(dev)
        P, _, it = b4.fwd(H, args.tol, args.max_iter, want_dual=False, want_iters=True)
        Psk = b4.sk_fwd(H, 20)
        torch.cuda.synchronize()
        row = {}
        for label, X in (("newton", P), ("sk20", Psk)):
            _, l1 = l1_stats(X)
            row[label] = [float(l1.mean().item()), float(l1.std().item()), float(l1.median().item()),
                          float(l1.max().item())]
        itn = it.cpu().numpy()
        row["newton_steps_mean"] = round(float(itn[itn >= 0].mean()), 3)
        row["newton_frac_over_20"] = float(((itn > PAPER_CAP) | (itn == -1)).mean())
        row["paper"] = PAPER_TABLES[name]
        out["families"][name] = row
        log(f"accuracy {name}: {row}")
    return out


def cpu_info() -> dict:
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        aff = len(os.sched_getaffinity(0))
    except AttributeError:
        aff = None
    return {"host_cpus": os.cpu_count(), "affinity_cpus": aff, "cpu_model": model}


def bench_cpu_baseline(args, ch, w) -> dict:
    """The oracle as it stands (fp64, its own tolerance 1e-13) on the headline workload's first
    matrices, fwd + bwd, on the host's CPU share of threads for one GPU; its 1-thread rate on a smaller sample
    at 1e-13 and at the GPU's tolerance; and the host's core count and CPU model."""
    import oracle
    n = min(args.cpu_sample, w.B)
    Hs = ch.H[:n].astype(np.float64)
    Gs = ch.dP[:n].astype(np.float64) if w.grad else None
    threads = oracle.default_threads()

    def rate(H, G, tol, nth):
        t0 = time.perf_counter()
        Pr, _, _ = oracle.fwd(H, tol=tol, threads=nth)
        if G is not None:
            oracle.bwd(Pr, G, threads=nth)
        dt = time.perf_counter() - t0
        return H.shape[0] / dt, dt

    v, dt = rate(Hs, Gs, oracle.DEFAULT_TOL, threads)
    vg, dtg = rate(Hs, Gs, args.tol, threads)
    n1 = min(n, 1 << 18)
    v1, dt1 = rate(Hs[:n1], Gs[:n1] if Gs is not None else None, oracle.DEFAULT_TOL, 1)
    v1g, dt1g = rate(Hs[:n1], Gs[:n1] if Gs is not None else None, args.tol, 1)
    info = cpu_info()
    res = {"value": round(v, 1), "unit": "proj/s", "cores": threads, "kind": "oracle",
           "sample": f"first {n} matrices of {w.name}; fp64 oracle forward (tol {oracle.DEFAULT_TOL:g}) + "
                     f"backward, {threads} threads (the host's CPU share for one GPU), {dt:.1f} s",
           **info,
           "at_gpu_tol": {"value": round(vg, 1), "tol": args.tol, "threads": threads, "seconds": round(dtg, 2)},
           "one_thread": {"value": round(v1, 1), "tol": oracle.DEFAULT_TOL, "sample": n1, "seconds": round(dt1, 2)},
           "one_thread_at_gpu_tol": {"value": round(v1g, 1), "tol": args.tol, "sample": n1,
                                     "seconds": round(dt1g, 2)}}
    log(f"cpu baseline: {res}")
    return res


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mix_bf16_b2e24")
    ap.add_argument("--tol", type=float, default=1e-6)
    ap.add_argument("--max-iter", type=int, default=64)
    ap.add_argument("--cpu-sample", type=int, default=1 << 24,
                    help="matrices in the oracle's CPU-baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sk", action="store_true")
    ap.add_argument("--no-hess", action="store_true", help="skip the saved-Hessian variant's timing")
    ap.add_argument("--no-configs", action="store_true", help="skip the other workload configurations")
    ap.add_argument("--no-n8", action="store_true", help="skip the 8x8 measurement")
    ap.add_argument("--n8-only", action="store_true", help="time only the 8x8 path (for profiler runs)")
    ap.add_argument("--no-ot", action="store_true", help="skip the general-OT measurement")
    ap.add_argument("--ot8-only", action="store_true", help="time only the 8x8 general-OT path (for profiler runs)")
    ap.add_argument("--ot-only", action="store_true", help="time only the general-OT path (for profiler runs)")
    ap.add_argument("--no-small", action="store_true", help="skip the small-batch launch timing")
    ap.add_argument("--no-mix", action="store_true", help="skip the residual-mixing measurement")
    ap.add_argument("--mix-only", action="store_true", help="time only the residual-mixing pair (for profiler runs)")
    ap.add_argument("--runtime-only", action="store_true", help="only the paper's runtime sweep (N(0,10^2), 0.5K-128K)")
    ap.add_argument("--small-only", action="store_true", help="time only the small-batch cases")
    ap.add_argument("--no-extras", action="store_true",
                    help="time only the given workload's path, none of the other measurements (for profiler runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy 5 times (scale for HBM byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: measures one GPU only; the projection shards by contiguous batch ranges with "
              "no communication between GPUs, so only --gpus 1 is measured.",
              file=sys.stderr)
        return 2

    import torch

    import workloads

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    if args.copy_calibration:
        X = torch.ones(1 << 28, device=dev)
        Y = torch.empty_like(X)
        for _ in range(5):
            Y.copy_(X)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration": {"bytes_read": X.numel() * 4, "bytes_written": Y.numel() * 4,
                                               "launches": 5}}), flush=True)
        return 0
    if args.n8_only:
        print(json.dumps({"n8": bench_n8(args, dev, stream)}), flush=True)
        return 0
    if args.ot_only:
        print(json.dumps({"ot": bench_ot(args, dev, stream)}), flush=True)
        return 0
    if args.mix_only:
        print(json.dumps({"mix_streams": bench_mix_streams(args, dev, stream),
                          "mix8_streams": bench_mix_streams(args, dev, stream, B=1 << 14, n=8)}), flush=True)
        return 0
    if args.small_only:
        print(json.dumps({"small_batch": bench_small_batch(dev)}), flush=True)
        return 0
    if args.runtime_only:
        print(json.dumps({"runtime_table": bench_runtime_table(args, dev, stream)}), flush=True)
        return 0
    if args.ot8_only:
        print(json.dumps({"ot8": bench_ot(args, dev, stream, n=8)}), flush=True)
        return 0

    w = workloads.WORKLOADS[args.workload]
    extras = not args.no_extras
    head = measure(w.name, args, dev, stream, extras=extras, sk=extras and not args.no_sk, buckets=extras,
                   autograd=extras, hess=extras and not args.no_hess)
    B, K = w.B, args.steps
    kernels = head["kernels"]
    dominant = max(kernels, key=lambda k: kernels[k]["avg_ms"])
    traffic = traffic_from_profiles(w.name)
    ach = kernels[dominant]["achieved_GBs"]
    roofline = {"bound": "hbm", "kernel": dominant, "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                "traffic": (traffic or {}).get(dominant)}
    # the forward is bound by its write requests and its VALU work together: its VALU issue
    # rate (lane-instructions counted by rocprofv3 on this source) is reported beside the bytes
    valu = valu_from_profiles(w.name, dominant, "traffic")
    if valu:
        va = valu / (kernels[dominant]["avg_ms"] * 1e-3) / 1e12
        roofline["valu"] = {"achieved": round(va, 2), "peak": VALU_PEAK_T, "unit": "T lane-instr/s",
                            "frac": round(va / VALU_PEAK_T, 4), "counted_lane_instr_per_launch": valu}
    out = {
        "metric": METRIC if w.name == "mix_bf16_b2e24" else f"4x4 Birkhoff projections/sec ({w.name})",
        "value": head["value"], "unit": "proj/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"], "fwd_proj_per_s": round(B / (head["_fwd_ms"] * 1e-3), 1),
        "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name, "B": B, "storage": w.storage, "tol": args.tol,
                   "max_iter": args.max_iter, "passes": head["passes"], "desc": w.desc,
                   "buffer_sets": head["buffer_sets"]},
        "roofline": roofline,
        "path_hbm_frac": head["path_hbm_frac"],
        "kernels": kernels,
    }
    for k in ("newton_steps", "max_marginal_err", "marginal_err_L1", "sk20_baseline", "buckets",
              "autograd_step", "saved_hessian"):
        if k in head:
            out[k] = head[k]
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = bench_cpu_baseline(args, head["_ch"], w)
    del head

    if extras and not args.no_configs:
        # the other workload configurations, each timed on its own after the headline's region
        cfg = {"n01_b4096": bench_b4096(args, dev)}
        for name, kw in (("n01_b2e20_fwd", {}), ("n10_b2e22", {"sk": True}),
                         ("logunif_b2e25", {"sk": True, "buckets": True}),
                         ("mix_bf16_b2e24", {"storage": "f32"})):
            r = measure(name, args, dev, stream, extras=True, **kw)
            cfg[r["workload"]] = public(r)
            del r
        out["configs"] = cfg
        out["accuracy_tables"] = bench_accuracy(args, dev)
        out["runtime_table"] = bench_runtime_table(args, dev, stream)
    if not args.no_n8 and extras:
        out["n8"] = bench_n8(args, dev, stream)
    if not args.no_ot and extras:
        out["ot"] = bench_ot(args, dev, stream)
        out["ot8"] = bench_ot(args, dev, stream, n=8)
    if not args.no_small and extras:
        out["small_batch"] = bench_small_batch(dev)
    if not args.no_mix and extras:
        out["mix_streams"] = bench_mix_streams(args, dev, stream)
        out["mix8_streams"] = bench_mix_streams(args, dev, stream, B=1 << 14, n=8)

    print(json.dumps(out), flush=True)
    return 0


def bench_mix_streams(args, dev, stream, B=1 << 15, C=4096, n=4) -> dict:
    """Residual mixing of the mHC layer (Y = P X per token, P = proj(exp(H))) and its backward
    on B tokens of 4 bf16 streams with C channels: per-call event times, algorithmic GB/s
    and the oracle's rate on a sample of tokens."""
    import torch

    import paper_2606_07574_amd as b4
    import workloads
    H, X, G = workloads.mix_streams_device(B, C, 60 + n, dev, n)
    Y = torch.empty_like(X)
    dX = torch.empty_like(X)
    P = torch.empty(B, n, n, device=dev)
    dH = torch.empty(B, n, n, device=dev)
    lib = b4.lib()
    mfwd, mbwd = (lib.birkhoff4_mix_fwd, lib.birkhoff4_mix_bwd) if n == 4 else (lib.birkhoff8_mix_fwd,
                                                                                 lib.birkhoff8_mix_bwd)
    sptr = stream.cuda_stream
    K = max(5, args.steps // 2)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]

    def step(e):
        if e:
            e[0].record(stream)
        rc = mfwd(H.data_ptr(), b4.BF16, X.data_ptr(), b4.BF16, Y.data_ptr(), P.data_ptr(), None, None, B, C,
                  args.tol, args.max_iter, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())
        if e:
            e[1].record(stream)
        rc = mbwd(P.data_ptr(), X.data_ptr(), G.data_ptr(), b4.BF16, dX.data_ptr(), dH.data_ptr(), B, C, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())
        if e:
            e[2].record(stream)
    for _ in range(2):
        step(None)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        step(ev[k])
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / K
    f_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    b_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    nn = n * n
    fb = 2 * nn + 4 * nn + 4 * n * C        # H (bf16), P, X, Y (bf16)
    bb = 4 * nn + 6 * n * C + 4 * nn        # P, X, dY, dX, dH
    name = f"mix_streams_b2e{B.bit_length() - 1}_c{C}" + ("" if n == 4 else f"_n{n}")
    res = {"workload": name, "B": B, "C": C, "n": n,
           "desc": f"B={B} tokens, {n} bf16 streams of C={C} channels, X, dY ~ N(0,1); logits H from the "
                   "headline mixture in bf16; fwd = projection + Y = P X, bwd = dX = P^T dY, dP = dY X^T, dH",
           "steps": K, "value": round(B / wall, 1), "unit": "tokens/s", "ms_per_step": round(wall * 1e3, 4),
           "fwd_ms": round(f_ms, 4), "bwd_ms": round(b_ms, 4),
           "alg_bytes_per_token": {"fwd": fb, "bwd": bb},
           "kernels": {"mix_fwd (projection + mixing)": {"achieved_GBs": round(B * fb / (f_ms * 1e-3) / 1e9, 1)},
                       "mix_bwd": {"achieved_GBs": round(B * bb / (b_ms * 1e-3) / 1e9, 1)}},
           "path_hbm_frac": round(B * (fb + bb) / wall / 1e9 / HBM_PEAK_GBS, 4)}
    # context: torch's own device copy of X into Y (the forward's stream bytes, no arithmetic)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    Y.copy_(X)
    c0.record(stream)
    for _ in range(K):
        Y.copy_(X)
    c1.record(stream)
    torch.cuda.synchronize()
    res["copy_reference_GBs"] = round(2 * X.numel() * 2 * K / (c0.elapsed_time(c1) * 1e-3) / 1e9, 1)
    dom = "mix_bwd" if b_ms >= f_ms else "mix_fwd (projection + mixing)"
    ach = res["kernels"][dom]["achieved_GBs"]
    res["roofline"] = {"bound": "hbm", "kernel": dom, "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                       "frac": round(ach / HBM_PEAK_GBS, 4),
                       # both stream counts are profiled in one file, the 4-stream workload's
                       "traffic": profile_figure(f"kernel_trace_mix_streams_b2e15_c{C}.md",
                                                 ("mix" if n == 4 else "mix8")
                                                 + ("_bwd" if dom == "mix_bwd" else "_fwd")
                                                 + "_hbm_bytes_per_launch")}
    log(f"mix streams: {res}")
    if not args.no_cpu_baseline:
        from oracle.mix import mix_bwd as o_bwd, mix_fwd as o_fwd
        import oracle
        n = 256
        Hs, Xs, Gs = H[:n].float().cpu().numpy(), X[:n].float().cpu().numpy(), G[:n].float().cpu().numpy()
        threads = oracle.default_threads()
        t0 = time.perf_counter()
        _, Pr = o_fwd(Hs, Xs, threads=threads)
        o_bwd(Pr, Xs, Gs, threads=threads)
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": round(n / dt, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
                               "sample": f"first {n} tokens of {res['workload']}; fp64 oracle (projection tol "
                                         f"{oracle.DEFAULT_TOL:g}, numpy products) fwd + bwd, {dt:.2f} s"}
    del H, X, G, Y, dX, P, dH
    return res


def bench_small_batch(dev, sizes=(512, 4096, 32768), pairs=32, reps=20, inputs=None) -> list:
    """Small batches are launch-bound: per fwd + bwd pair (N(0,1) logits, fp32, default
    variant), the wall time of back-to-back eager calls, the same pairs replayed from a HIP
    graph that holds `pairs` of them, and the two kernels' event-timed durations."""
    import torch

    import paper_2606_07574_amd as b4
    import workloads
    res = []
    for B in sizes:
        H32, dP32 = inputs[B] if inputs and B in inputs else workloads.gauss(B, 1.0, seed=B)
        H = torch.from_numpy(H32).to(dev)
        dP = torch.from_numpy(dP32).to(dev)
        P = torch.empty_like(H)
        dH = torch.empty_like(H)

        def pair():
            b4.fwd(H, out=P, want_dual=False)
            b4.bwd(P, dP, out=dH)
        for _ in range(20):
            pair()
        torch.cuda.synchronize()
        n = pairs * reps
        t0 = time.perf_counter()
        for _ in range(n):
            pair()
        torch.cuda.synchronize()
        eager_us = (time.perf_counter() - t0) / n * 1e6
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(pairs):
                pair()
        for _ in range(2):
            g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            g.replay()
        torch.cuda.synchronize()
        graph_us = (time.perf_counter() - t0) / n * 1e6
        stream = torch.cuda.current_stream(dev)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        f_ms = b_ms = 0.0
        for _ in range(reps):
            ev[0].record(stream)
            b4.fwd(H, out=P, want_dual=False)
            ev[1].record(stream)
            b4.bwd(P, dP, out=dH)
            ev[2].record(stream)
            torch.cuda.synchronize()
            f_ms += ev[0].elapsed_time(ev[1])
            b_ms += ev[1].elapsed_time(ev[2])
        row = {"B": B, "eager_us_per_pair": round(eager_us, 2), "graph_us_per_pair": round(graph_us, 2),
               "pairs_per_graph": pairs, "fwd_event_us": round(f_ms / reps * 1e3, 2),
               "bwd_event_us": round(b_ms / reps * 1e3, 2),
               "graph_proj_per_s": round(B / (graph_us * 1e-6), 1)}
        log(f"small batch: {row}")
        res.append(row)
        del g, H, dP, P, dH
    return res


def bench_autograd_step(args, lib, sets, n_sets, B, hcode, bf16, stream, inb) -> dict:
    """The step that autograd runs (project(): the forward without the dual, which the backward
    does not read, then the backward) on the benchmark's buffers, timed like the headline."""
    import torch

    import paper_2606_07574_amd as b4
    sptr = stream.cuda_stream
    gcode = hcode if bf16 else b4.F32
    K = args.steps
    e0 = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
    e1 = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
    e2 = [torch.cuda.Event(enable_timing=True) for _ in range(K)]

    def step(k, ev):
        st = sets[k % n_sets]
        if ev:
            e0[k].record(stream)
        rc = lib.birkhoff4_fwd_ex(st["H"].data_ptr(), hcode, st["P"].data_ptr(), None, None, B, args.tol,
                                  args.max_iter, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())
        if ev:
            e1[k].record(stream)
        rc = lib.birkhoff4_bwd_ex(st["P"].data_ptr(), st["G"].data_ptr(), gcode, st["dH"].data_ptr(), B, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())
        if ev:
            e2[k].record(stream)
    for k in range(args.warmup):
        step(k, False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        step(k, True)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / K
    f_ms = float(np.mean([e0[k].elapsed_time(e1[k]) for k in range(K)]))
    b_ms = float(np.mean([e1[k].elapsed_time(e2[k]) for k in range(K)]))
    fb, bb = inb + 64, 64 + inb + 64
    return {"ms_per_step": round(wall * 1e3, 4), "value": round(B / wall, 1), "unit": "proj/s",
            "fwd_ms": round(f_ms, 4), "bwd_ms": round(b_ms, 4), "alg_bytes_per_projection": fb + bb,
            "fwd_GBs": round(B * fb / (f_ms * 1e-3) / 1e9, 1), "bwd_GBs": round(B * bb / (b_ms * 1e-3) / 1e9, 1),
            "path_hbm_frac": round(B * (fb + bb) / wall / 1e9 / HBM_PEAK_GBS, 4)}


def bench_saved_hessian(args, lib, sets, n_sets, B, hcode, bf16, stream, inb, default_ms):
    """The saved-Hessian variant (Sec. 4.2) on the benchmark's buffers: the forward also writes
    the 32-byte column weights of P, the backward reads them instead of recomputing them."""
    import torch

    import paper_2606_07574_amd as b4
    dev = sets[0]["H"].device
    hs = [torch.empty(B, 8, device=dev) for _ in range(n_sets)]
    sptr = stream.cuda_stream
    gcode = hcode if bf16 else b4.F32
    ks = max(3, args.steps // 2)
    e0 = [torch.cuda.Event(enable_timing=True) for _ in range(ks)]
    e1 = [torch.cuda.Event(enable_timing=True) for _ in range(ks)]
    e2 = [torch.cuda.Event(enable_timing=True) for _ in range(ks)]

    def step(k, ev):
        st, h = sets[k % n_sets], hs[k % n_sets]
        if ev:
            e0[k].record(stream)
        rc = lib.birkhoff4_fwd_hess(st["H"].data_ptr(), hcode, st["P"].data_ptr(), st["dual"].data_ptr(),
                                    h.data_ptr(), None, B, args.tol, args.max_iter, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())
        if ev:
            e1[k].record(stream)
        rc = lib.birkhoff4_bwd_hess(st["P"].data_ptr(), h.data_ptr(), st["G"].data_ptr(), gcode,
                                    st["dH"].data_ptr(), B, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())
        if ev:
            e2[k].record(stream)

    for k in range(2):
        step(k, False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(ks):
        step(k, True)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / ks
    f_ms = float(np.mean([e0[k].elapsed_time(e1[k]) for k in range(ks)]))
    b_ms = float(np.mean([e1[k].elapsed_time(e2[k]) for k in range(ks)]))
    fwd_bytes, bwd_bytes = B * (inb + 64 + 32 + 32), B * (64 + 32 + inb + 64)
    return {"ms_per_step": round(wall * 1e3, 4), "value": round(B / wall, 1), "unit": "proj/s",
            "fwd_ms": round(f_ms, 4), "bwd_ms": round(b_ms, 4),
            "alg_bytes_per_projection": (fwd_bytes + bwd_bytes) // B,
            "fwd_GBs": round(fwd_bytes / (f_ms * 1e-3) / 1e9, 1), "bwd_GBs": round(bwd_bytes / (b_ms * 1e-3) / 1e9, 1),
            "default_ms_per_step": round(default_ms, 4)}


def bucket_report(w, ch, itn, marg, sk_marg):
    """Newton steps and max marginal error (and the SK-20 baseline's) per input bucket: the
    mixture's four kinds, deciles of the log-uniform scale, or the one Gaussian scale."""
    if w.kind == "mixture":
        sel = [(f"gauss sigma={sg:g}", (ch.kind == 0) & (ch.scale == np.float32(sg))) for sg in (1.0, 5.0, 20.0)]
        sel.append(("near-permutation 20 Pi + 0.1 N", ch.kind == 1))
    elif w.kind == "logunif":
        edges = np.quantile(ch.scale, np.linspace(0.0, 1.0, 11))
        sel = []
        for d in range(10):
            lo, hi = edges[d], edges[d + 1]
            m = (ch.scale >= lo) & ((ch.scale < hi) if d < 9 else (ch.scale <= hi))
            sel.append((f"alpha decile {d + 1}: [{lo:.3g}, {hi:.3g}]", m))
    else:
        sel = [(f"sigma={w.sigma:g}", np.ones(len(itn), bool))]
    rows = []
    for name, m in sel:
        it = itn[m]
        conv = it[it >= 0]
        row = {"bucket": name, "n": int(m.sum()),
               "newton_steps": {"mean": round(float(conv.mean()), 3) if len(conv) else None,
                                "p99": int(np.percentile(conv, 99)) if len(conv) else None,
                                "max": int(conv.max()) if len(conv) else None,
                                "not_converged": int((it == -1).sum()),
                                "hist": np.bincount(np.clip(conv, 0, 40), minlength=41).tolist()},
               "max_marginal_err": float(marg[m].max()) if m.any() else None}
        if sk_marg is not None and m.any():
            row["sk20_max_marginal_err"] = float(sk_marg[m].max())
            row["sk20_median_marginal_err"] = float(np.median(sk_marg[m]))
        rows.append(row)
    return rows


OT_B = 1 << 22
OT_ETA = 0.5
OT_DESC = ("B=2^22 4x4 entropic OT problems, fp32: cost M = 2 N(0,1), marginals a, b ~ U(0.2, 2) with b rescaled "
           "to sum(a), eta = 0.5; dT ~ N(0,1); fwd + bwd")


def bench_ot(args, dev, stream, n: int = 4) -> dict:
    """fwd + bwd of n x n entropic OT with general marginals (n = 4 or 8; reported beside the
    4x4 path)."""
    import torch

    import paper_2606_07574_amd as b4
    import workloads
    B = OT_B
    name = "ot_b2e22" if n == 4 else "ot8_b2e22"
    kf, kb = ("ot4_fwd", "ot4_bwd") if n == 4 else ("ot8_fwd", "ot8_bwd")
    M, a, b, G = workloads.ot_device(B, 4 if n == 4 else 48, dev, n)
    T = torch.empty(B, n, n, device=dev)
    dual = torch.empty(B, 2 * n, device=dev)
    dM = torch.empty(B, n, n, device=dev)
    lib = b4.lib()
    fwd_fn = lib.birkhoff4_ot_fwd if n == 4 else lib.birkhoff8_ot_fwd
    bwd_fn = lib.birkhoff4_ot_bwd if n == 4 else lib.birkhoff8_ot_bwd
    sptr = stream.cuda_stream

    def step():
        rc = fwd_fn(M.data_ptr(), a.data_ptr(), b.data_ptr(), OT_ETA, T.data_ptr(), dual.data_ptr(),
                    None, B, args.tol, args.max_iter, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())
        e_mid.record(stream)
        rc = bwd_fn(T.data_ptr(), a.data_ptr(), G.data_ptr(), OT_ETA, dM.data_ptr(), B, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())

    K = max(3, args.steps // 4)
    e0, e_mid, e1 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    step()
    torch.cuda.synchronize()
    f_ms = b_ms = 0.0
    for _ in range(K):
        e0.record(stream)
        step()
        e1.record(stream)
        torch.cuda.synchronize()
        f_ms += e0.elapsed_time(e_mid)
        b_ms += e_mid.elapsed_time(e1)
    f_ms /= K
    b_ms /= K
    nn, nv = 4 * n * n, 4 * n  # bytes of a matrix and of a marginal
    fwd_bytes = B * (nn + 2 * nv + nn + 2 * nv)
    bwd_bytes = B * (nn + nv + nn + nn)
    res = {"workload": name, "B": B, "n": n, "eta": OT_ETA, "desc": OT_DESC.replace("4x4", f"{n}x{n}"), "steps": K,
           "value": round(B / ((f_ms + b_ms) * 1e-3), 1), "unit": "problems/s",
           "fwd_ms": round(f_ms, 4), "bwd_ms": round(b_ms, 4),
           "kernels": {kf: {"alg_bytes_per_launch": fwd_bytes,
                            "achieved_GBs": round(fwd_bytes / (f_ms * 1e-3) / 1e9, 1)},
                       kb: {"alg_bytes_per_launch": bwd_bytes,
                            "achieved_GBs": round(bwd_bytes / (b_ms * 1e-3) / 1e9, 1)}},
           "path_hbm_frac": round((fwd_bytes + bwd_bytes) / ((f_ms + b_ms) * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    valu = valu_from_profiles(name, kf, "kernel_trace")
    ach = valu / (f_ms * 1e-3) / 1e12 if valu else None
    res["roofline"] = {"bound": "alu", "kernel": kf,
                       "achieved": round(ach, 2) if ach else None, "peak": VALU_PEAK_T,
                       "unit": "T lane-instr/s", "frac": round(ach / VALU_PEAK_T, 4) if ach else None,
                       "counted_lane_instr_per_launch": valu}
    if args.ot_only or args.ot8_only:
        return res
    _, _, it = (b4.ot_fwd if n == 4 else b4.ot8_fwd)(M, a, b, OT_ETA, args.tol, args.max_iter, want_dual=False,
                                                       want_iters=True)
    torch.cuda.synchronize()
    itn = it.cpu().numpy()
    conv = itn[itn >= 0]
    T64 = T.double()
    res["newton_steps"] = {"mean": round(float(conv.mean()), 3), "p99": int(np.percentile(conv, 99)),
                           "max": int(conv.max()), "not_converged": int((itn == -1).sum()),
                           "non_finite": int((itn == -2).sum())}
    res["max_marginal_err"] = float(torch.maximum((T64.sum(-1) - a.double()).abs().amax(),
                                                  (T64.sum(-2) - b.double()).abs().amax()).item())
    del T64
    log(f"{name}: {res['value']:.4g} problems/s fwd {f_ms:.3f} ms bwd {b_ms:.3f} ms; steps {res['newton_steps']}; "
        f"max marginal {res['max_marginal_err']:.3e}")
    if not args.no_cpu_baseline:
        from oracle import birkhoffn
        ns = 1 << 20 if n == 4 else 1 << 18
        Ms, As, Bs, Gs = (x[:ns].double().cpu().numpy() for x in (M, a, b, G))
        Bs = Bs * (As.sum(1) / Bs.sum(1))[:, None]
        threads = max(1, min(16, os.cpu_count() or 1))
        t0 = time.perf_counter()
        Tr, _, _ = birkhoffn.ot_fwd(Ms, As, Bs, OT_ETA, threads=threads)
        birkhoffn.ot_bwd(Tr, As, Gs, OT_ETA, threads=threads)
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": round(ns / dt, 1), "unit": "problems/s", "cores": threads, "kind": "oracle",
                               "sample": f"first {ns} problems of {name}; fp64 OT oracle forward (tol "
                                         f"{birkhoffn.DEFAULT_TOL:g}) + backward, {threads} threads, {dt:.1f} s"}
        log(f"{name} cpu baseline: {res['cpu_baseline']}")
    return res


N8_B = 1 << 22
N8_DESC = ("B=2^22 8x8 matrices, bf16 storage, fp32 compute; half sigma*N(0,1) with sigma in {1,5,20}, "
           "half 20*Pi + 0.1 N(0,1) (Pi a random permutation); dP ~ N(0,1) bf16; fwd + bwd")


def bench_n8(args, dev, stream) -> dict:
    """fwd + bwd of the 8x8 projection on its mixture workload (reported beside the 4x4 path)."""
    import torch

    import paper_2606_07574_amd as b4
    import workloads
    B = N8_B
    H, G = workloads.n8_mix_device(B, 8, dev)
    P = torch.empty(B, 8, 8, device=dev)
    dual = torch.empty(B, 16, device=dev)
    dH = torch.empty(B, 8, 8, device=dev)
    lib = b4.lib()
    sptr = stream.cuda_stream

    def step():
        rc = lib.birkhoff8_fwd(H.data_ptr(), b4.BF16, P.data_ptr(), dual.data_ptr(), None, B, args.tol,
                               args.max_iter, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())
        e_mid.record(stream)
        rc = lib.birkhoff8_bwd(P.data_ptr(), G.data_ptr(), b4.BF16, dH.data_ptr(), B, sptr)
        if rc:
            raise RuntimeError(lib.birkhoff4_strerror(rc).decode())

    K = max(3, args.steps // 4)
    e0, e_mid, e1 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    step()
    torch.cuda.synchronize()
    f_ms = b_ms = 0.0
    t_start = time.perf_counter()
    for _ in range(K):
        e0.record(stream)
        step()
        e1.record(stream)
        torch.cuda.synchronize()
        f_ms += e0.elapsed_time(e_mid)
        b_ms += e_mid.elapsed_time(e1)
    wall = time.perf_counter() - t_start
    f_ms /= K
    b_ms /= K
    fwd_bytes = B * (128 + 256 + 64)
    bwd_bytes = B * (256 + 128 + 256)
    res = {"workload": "n8_mix_bf16_b2e22", "B": B, "desc": N8_DESC, "steps": K,
           "value": round(B / ((f_ms + b_ms) * 1e-3), 1), "unit": "proj/s",
           "ms_per_step": round(wall * 1e3 / K, 4), "fwd_ms": round(f_ms, 4), "bwd_ms": round(b_ms, 4),
           "kernels": {"newton8_fwd": {"alg_bytes_per_launch": fwd_bytes,
                                       "achieved_GBs": round(fwd_bytes / (f_ms * 1e-3) / 1e9, 1)},
                       "implicit8_bwd": {"alg_bytes_per_launch": bwd_bytes,
                                         "achieved_GBs": round(bwd_bytes / (b_ms * 1e-3) / 1e9, 1)}},
           "path_hbm_frac": round((fwd_bytes + bwd_bytes) / ((f_ms + b_ms) * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    valu = valu_from_profiles("n8_mix_bf16_b2e22", "newton8_fwd")
    ach = valu / (f_ms * 1e-3) / 1e12 if valu else None
    res["roofline"] = {"bound": "alu", "kernel": "newton8_fwd",
                       "achieved": round(ach, 2) if ach else None, "peak": VALU_PEAK_T,
                       "unit": "T lane-instr/s", "frac": round(ach / VALU_PEAK_T, 4) if ach else None,
                       "counted_lane_instr_per_launch": valu}
    if args.n8_only:
        return res
    _, _, it = b4.fwd8(H, args.tol, args.max_iter, want_dual=False, want_iters=True)
    torch.cuda.synchronize()
    itn = it.cpu().numpy()
    P64 = P.double()
    marg = torch.maximum((P64.sum(-1) - 1).abs().amax(-1), (P64.sum(-2) - 1).abs().amax(-1))
    conv = itn[itn >= 0]
    n64 = (len(itn) // 64) * 64
    res["newton_steps"] = {"mean": round(float(conv.mean()), 3), "p99": int(np.percentile(conv, 99)),
                           "max": int(conv.max()),
                           "mean_of_wave_max": round(float(np.clip(itn[:n64], 0, None).reshape(-1, 64)
                                                           .max(axis=1).mean()), 3),
                           "not_converged": int((itn == -1).sum()), "non_finite": int((itn == -2).sum())}
    res["max_marginal_err"] = float(marg.max().item())
    del P64
    log(f"n8: {res['value']:.4g} proj/s fwd {f_ms:.3f} ms bwd {b_ms:.3f} ms; steps {res['newton_steps']}; "
        f"max marginal {res['max_marginal_err']:.3e}")
    if not args.no_cpu_baseline:
        from oracle import birkhoffn
        n = 1 << 20
        Hs = H[:n].float().cpu().numpy().astype(np.float64)
        Gs = G[:n].float().cpu().numpy().astype(np.float64)
        threads = max(1, min(16, os.cpu_count() or 1))
        t0 = time.perf_counter()
        Pr, _, _ = birkhoffn.fwd(Hs, threads=threads)
        birkhoffn.bwd(Pr, Gs, threads=threads)
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": round(n / dt, 1), "unit": "proj/s", "cores": threads, "kind": "oracle",
                               "sample": f"first {n} matrices of n8_mix_bf16_b2e22; fp64 size-generic oracle "
                                         f"forward (tol {birkhoffn.DEFAULT_TOL:g}) + backward, {threads} threads, "
                                         f"{dt:.1f} s"}
        log(f"n8 cpu baseline: {res['cpu_baseline']}")
    return res


if __name__ == "__main__":
    sys.exit(main())
