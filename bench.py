#!/usr/bin/env python3
"""Benchmark: BF16 attention forward + GProj backward on one MI355X.

One step = the whole hot path on one batch: FA3-SBS forward (O, LSE), then the
backward in gproj mode (preprocess, query-major pass with the query
correction, key-major pass with the key correction).  Workload: B=1, H=16,
N=4096, d=64, causal, alpha = 1/8, seeded synthetic inputs with a per-channel
key bias ~ N(0, 4^2) shared by all tokens and dO ~ N(0, 0.01^2).

Prints one JSON line.  value = fwd+bwd TFLOP/s with the FlashAttention count
7 * d * N^2 * B * H (causal pairs counted as N^2/2; forward 2 and backward 5
GEMM-equivalents), the same count in every mode.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "attn fwd+bwd TFLOP/s at H16 N4096 d64 causal; dQ/dK/dV rel-L2 vs FP64"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
NOMINAL_CLOCK_GHZ = 2.4     # the clock the published peaks assume
PEAK_HBM_GBS = 8000.0
PEAK_FP32_TFLOPS = 157.3    # MI355X FP32 (vector and matrix)

# Dense contractions per causal (query, key) pair that each kernel forms first
# (algorithmic), and that it executes (algorithmic + recompute), per mode.
ALG_PRODUCTS = {"fwd_sbs": {"plain": 2, "gproj_q": 2, "gproj": 2},
                "bwd_dq": {"plain": 3, "gproj_q": 4, "gproj": 4},        # S, dP, tK (+ rK)
                "bwd_dkdv": {"plain": 2, "gproj_q": 2, "gproj": 3}}      # r^T dO, t^T Q (+ r^T z)
EXEC_PRODUCTS = {"fwd_sbs": ALG_PRODUCTS["fwd_sbs"], "bwd_dq": ALG_PRODUCTS["bwd_dq"],
                 "bwd_dkdv": {m: p + 2 for m, p in ALG_PRODUCTS["bwd_dkdv"].items()}}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    # The part needs some tens of milliseconds of sustained load to reach its
    # steady clock; 200 warmup steps (~45 ms at the default size) get there,
    # and 200 timed steps take ~45 ms.
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=200)
    p.add_argument("--mode", default="gproj", choices=["plain", "gproj_q", "gproj"])
    p.add_argument("--workload", default="h16_n4096_d64",
                   help="synthetic workload to time (h16_n4096_d64 is the reference one; "
                        "others: tiny, h16_n4096_d128, h16_n16384_d64, b8_h32_n8192_d128)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-accuracy", action="store_true")
    p.add_argument("--no-configs", action="store_true",
                   help="skip the timing of the d = 128, long-sequence and batched workloads")
    p.add_argument("--no-seeds", action="store_true",
                   help="skip the 8-seed accuracy protocol of the reference workload")
    p.add_argument("--no-gqa", action="store_true",
                   help="skip the timing of the grouped-query layout (16 query / 4 key-value heads)")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="also run a cache-cold 512 MiB device copy (reference for HBM byte counters)")
    return p.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_h16_n4096_d64.json")
KERNEL_SOURCES = ["paper_2609_34272_amd/csrc/gpa_bwd.hip", "paper_2609_34272_amd/csrc/gpa_fwd.hip",
                  "paper_2609_34272_amd/csrc/gpa_device.h"]


def kernel_source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel: str, mode: str, workload: str = "h16_n4096_d64"):
    """HBM bytes per launch of `kernel` from the committed PMC summary, or None
    if there is none for this workload or the kernel sources changed since it
    was taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_digest") != kernel_source_digest() or rec.get("workload") != workload:
        return None
    k = rec.get("kernels", {}).get(f"{kernel}/{mode}")
    return None if k is None else k.get("hbm_bytes_per_launch")


def recorded_clock(kernel: str, mode: str, workload: str = "h16_n4096_d64"):
    """The clock (GHz) `kernel` ran at in the committed counter pass, or None
    (no record for this workload, or the kernel sources changed since)."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_digest") != kernel_source_digest() or rec.get("workload") != workload:
        return None
    k = rec.get("kernels", {}).get(f"{kernel}/{mode}")
    return None if k is None else k.get("clock_ghz")


def time_config(gpa, S, wc, seed, iters, dev, to_dev, oracle=None, heads=None):
    """Forward and per-mode backward times of one multi-head workload (mean of
    `iters` calls after ~100 ms of load, and the p10 / median / p90 of `iters`
    individually timed calls), its fwd+bwd TFLOP/s by the standard
    count, the GProj overhead and every kernel's fraction of the bf16 peak by
    its algorithmic products.  With the oracle, also the relative L2 errors
    (%) of O, dQ, dK, dV in every mode and of the FP32 baseline against the
    FP64 VJP, over the whole tensors or over the listed (b, h) heads."""
    import torch
    xc = S.make_inputs(wc, seed, workers=16)
    q, k, v, u = (to_dev(xc[n]) for n in ("q", "k", "v", "do"))
    if oracle is None:
        del xc
    B, H, N, d = wc.B, wc.H, wc.N, wc.d

    def timed(fn):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters

    def per_call(fn):
        # p10 / median / p90 of `iters` calls, each between its own events
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(iters)]
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        t = sorted(a.elapsed_time(b) for a, b in ev)
        q = lambda f: t[min(len(t) - 1, int(round(f * (len(t) - 1))))]  # noqa: E731
        return [round(q(0.1), 5), round(q(0.5), 5), round(q(0.9), 5)]

    o, lse = gpa.attn_fwd(q, k, v, wc.causal, wc.scale)
    # keep the GPU busy for ~100 ms first, so every mode is timed at the same
    # sustained clock
    wsw = torch.empty(gpa.attn_bwd_workspace_bytes(B, H, N, d, "gproj"), dtype=torch.uint8,
                      device=dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 0.1:
        gpa.attn_bwd(q, k, v, o, lse, u, "gproj", wc.causal, wc.scale, workspace=wsw)
        torch.cuda.synchronize()
    del wsw
    fwd = lambda: gpa.attn_fwd(q, k, v, wc.causal, wc.scale)  # noqa: E731
    res = {"B": B, "H": H, "N": N, "d": d, "seed": seed, "calls_timed": iters,
           "fwd_ms": round(timed(fwd), 5), "bwd_ms": {}, "kernel_frac": {},
           "per_call_ms_p10_p50_p90": {"fwd": per_call(fwd)}}
    pairs = B * H * N * N / 2.0
    for m in gpa.MODES:
        ws = torch.empty(gpa.attn_bwd_workspace_bytes(B, H, N, d, m), dtype=torch.uint8, device=dev)
        fn = lambda: gpa.attn_bwd(q, k, v, o, lse, u, m, wc.causal, wc.scale, workspace=ws)  # noqa: E731
        res["bwd_ms"][m] = round(timed(fn), 5)
        res["per_call_ms_p10_p50_p90"]["bwd_" + m] = per_call(fn)
        gpa.profile_enable(True)
        for _ in range(iters):
            fn()
        torch.cuda.synchronize()
        prof = gpa.profile_read()
        gpa.profile_enable(False)
        for name, (tot, cnt) in prof.items():
            if cnt and name in ALG_PRODUCTS:
                t = tot / cnt
                res["kernel_frac"][f"{name}/{m}"] = {
                    "avg_ms": round(t, 5),
                    "frac": round(ALG_PRODUCTS[name][m] * 2.0 * d * pairs / (t * 1e-3) / 1e12
                                  / PEAK_BF16_TFLOPS, 4)}
        del ws
    gpa.profile_enable(True)
    for _ in range(iters):
        gpa.attn_fwd(q, k, v, wc.causal, wc.scale)
    torch.cuda.synchronize()
    prof = gpa.profile_read()
    gpa.profile_enable(False)
    tot, cnt = prof["fwd_sbs"]
    res["kernel_frac"]["fwd_sbs"] = {"avg_ms": round(tot / cnt, 5),
                                     "frac": round(2 * 2.0 * d * pairs / (tot / cnt * 1e-3) / 1e12
                                                   / PEAK_BF16_TFLOPS, 4)}
    flops = 7.0 * d * N * N * B * H
    res["fwd_bwd_tflops_gproj"] = round(flops / ((res["fwd_ms"] + res["bwd_ms"]["gproj"]) * 1e-3)
                                        / 1e12, 2)
    res["gproj_bwd_overhead_vs_plain_pct"] = round(
        100.0 * (res["bwd_ms"]["gproj"] / res["bwd_ms"]["plain"] - 1), 2)
    res["gproj_q_bwd_overhead_vs_plain_pct"] = round(
        100.0 * (res["bwd_ms"]["gproj_q"] / res["bwd_ms"]["plain"] - 1), 2)
    if oracle is not None:
        import numpy as np
        sel = list(heads) if heads else [(b, h) for b in range(B) for h in range(H)]
        bi = torch.tensor([b for b, _ in sel], device=dev)
        hi = torch.tensor([h for _, h in sel], device=dev)
        host = lambda t: t[bi, hi].float().cpu().numpy().astype(np.float64)  # noqa: E731
        outs = {}
        for m in gpa.MODES:
            dq, dk, dv = gpa.attn_bwd(q, k, v, o, lse, u, m, wc.causal, wc.scale)
            outs[m] = [host(t) for t in (o, dq, dk, dv)]
            del dq, dk, dv
        fo, _, fdq, fdk, fdv = gpa.fp32_attn(q, k, v, u, wc.causal, wc.scale)
        outs["fp32"] = [host(t) for t in (fo, fdq, fdk, fdv)]
        del fo, fdq, fdk, fdv
        pick = lambda a: np.stack([a[b, h] for b, h in sel])  # noqa: E731
        ex = oracle.exact(pick(xc["q"]), pick(xc["k"]), pick(xc["v"]), pick(xc["do"]), wc.causal,
                          wc.scale)
        res["rel_l2_pct_vs_fp64"] = {
            "heads": "all" if not heads else [list(p) for p in sel],
            **{m: {n: round(oracle.rel_l2(t, ex[n]), 4) for n, t in zip(("O", "dQ", "dK", "dV"), ts)}
               for m, ts in outs.items()}}
        del xc
    del q, k, v, u, o, lse
    torch.cuda.empty_cache()
    return res


def seed_protocol(gpa, S, oracle, w, index, to_dev):
    """Accuracy over the eight seeds 1000*index + s (s = 0..7) of a workload:
    per-seed and median full-tensor relative L2 (%) against the FP64 oracle
    for O, dQ, dK, dV in every mode and for the FP32 baseline (the paper
    reports medians over its eight captures)."""
    import numpy as np
    import torch
    seeds = S.seeds_for(index, 8)
    names = ("O", "dQ", "dK", "dV")
    per = {m: {n: [] for n in names} for m in (*gpa.MODES, "fp32")}
    for seed in seeds:
        x = S.make_inputs(w, seed, workers=16)
        q, k, v, u = (to_dev(x[n]) for n in ("q", "k", "v", "do"))
        o, lse = gpa.attn_fwd(q, k, v, w.causal, w.scale)
        res = {m: (o, *gpa.attn_bwd(q, k, v, o, lse, u, m, w.causal, w.scale)) for m in gpa.MODES}
        fo, _, fdq, fdk, fdv = gpa.fp32_attn(q, k, v, u, w.causal, w.scale)
        res["fp32"] = (fo, fdq, fdk, fdv)
        torch.cuda.synchronize()
        ex = oracle.exact(x["q"], x["k"], x["v"], x["do"], w.causal, w.scale)
        for m, ts in res.items():
            for n, t in zip(names, ts):
                per[m][n].append(round(oracle.rel_l2(
                    t.float().cpu().numpy().astype(np.float64), ex[n]), 4))
    return {"workload": w.name, "seeds": seeds, "per_seed": per,
            "median": {m: {n: round(float(np.median(vals)), 4) for n, vals in d_.items()}
                       for m, d_ in per.items()}}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(f"bench.py: runs on one GPU only (asked for {args.gpus}); "
              "the attention path shards over (batch, head) with no exchange, so per-GPU "
              "throughput is the single-GPU figure.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_34272_amd as gpa
    import synthetic as S

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    gpa.lib()
    dev = torch.device("cuda:0")
    wid = {wl.name: i for i, wl in S.WORKLOADS.items()}
    if args.workload not in wid or S.WORKLOADS[wid[args.workload]].kv_heads != S.WORKLOADS[wid[args.workload]].H:
        print(f"bench.py: unknown multi-head workload {args.workload!r}", file=sys.stderr)
        sys.exit(2)
    w = S.WORKLOADS[wid[args.workload]]
    B, H, N, d = w.B, w.H, w.N, w.d
    seed = 1000 * wid[args.workload]
    x = S.make_inputs(w, seed)

    def to_dev(b):
        return torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).view(torch.bfloat16).to(dev)

    q, k, v, u = (to_dev(x[n]) for n in ("q", "k", "v", "do"))
    ws = {m: torch.empty(gpa.attn_bwd_workspace_bytes(B, H, N, d, m), dtype=torch.uint8, device=dev)
          for m in gpa.MODES}
    flops = 7.0 * d * N * N * B * H / 1.0  # FA convention: causal pairs N^2/2, 14 d per pair

    def step(mode):
        o, lse = gpa.attn_fwd(q, k, v, w.causal, w.scale)
        return gpa.attn_bwd(q, k, v, o, lse, u, mode, w.causal, w.scale, workspace=ws[mode])

    def timed(fn, iters):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters

    for _ in range(args.warmup):
        step(args.mode)
    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    ms = timed(lambda: step(args.mode), args.steps)
    wall = time.perf_counter() - t_wall0
    value = flops / (ms * 1e-3) / 1e12

    # Per-kernel durations (HIP events that each kernel launch records at the
    # kernel's start and end on its stream).
    gpa.profile_enable(True)
    for _ in range(args.steps):
        step(args.mode)
    torch.cuda.synchronize()
    prof = gpa.profile_read()
    gpa.profile_enable(False)
    kern = {name: (tot / cnt if cnt else 0.0) for name, (tot, cnt) in prof.items() if cnt}

    # Backward alone per mode (for the GProj overhead over the plain backward),
    # in interleaved rounds, each mode keeping its fastest round: timed one
    # after the other, the first mode would fall in the clock transient that
    # follows the timed steps and flatter the overhead.
    o, lse = gpa.attn_fwd(q, k, v, w.causal, w.scale)
    bwd_ms = {}
    for _ in range(3):
        for m in gpa.MODES:
            fm = (lambda m_: lambda: gpa.attn_bwd(q, k, v, o, lse, u, m_, w.causal, w.scale,
                                                  workspace=ws[m_]))(m)
            for _ in range(3):
                fm()
            t = timed(fm, args.steps)
            bwd_ms[m] = min(bwd_ms.get(m, t), t)
    # Algorithm 1's own schedule (one key-major pass with FP32 atomic
    # accumulation of the query-side sums; gproj adds the key-correction
    # pass): for plain the other candidate for the fastest plain backward, for
    # the GProj modes the literal schedule beside the two-pass one.
    atomic_kern = {}
    for m in gpa.MODES:
        wsa = torch.empty(gpa.attn_bwd_atomic_workspace_bytes(B, H, N, d, m), dtype=torch.uint8,
                          device=dev)
        fa = lambda: gpa.attn_bwd_atomic(q, k, v, o, lse, u, m, w.causal, w.scale,  # noqa: E731
                                         workspace=wsa)
        for _ in range(3):
            fa()
        bwd_ms["plain_atomic_dq" if m == "plain" else m + "_atomic"] = timed(fa, args.steps)
        gpa.profile_enable(True)
        for _ in range(max(5, args.steps // 5)):
            fa()
        torch.cuda.synchronize()
        aprof = gpa.profile_read()
        gpa.profile_enable(False)
        atomic_kern[m] = {n: round(t / c, 5) for n, (t, c) in aprof.items() if c}
        del wsa
    fwd_ms = timed(lambda: gpa.attn_fwd(q, k, v, w.causal, w.scale), args.steps)
    # Reference only (not `value`): the same K steps timed after 200 further
    # steps of this workload.  From idle the part runs its first milliseconds
    # at a boost clock and then throttles for several milliseconds before it
    # settles (kernel traces show the key pass at ~91 us in the first steps,
    # 100-110 us in the next ones and ~88 us once settled), and each switch to
    # another heavy workload starts a new transient; a short run times the
    # transient, a training loop runs at the settled clock.
    for _ in range(200):
        step(args.mode)
    ms_steady = timed(lambda: step(args.mode), args.steps)

    # Per-call distribution (p10 / median / p90 ms): each call bracketed by its
    # own pair of events, so each figure carries a few microseconds of event
    # overhead that the K-step means above do not.
    def percentiles(fn, iters):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(iters)]
        torch.cuda.synchronize()
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        t = np.sort(np.array([a.elapsed_time(b) for a, b in ev]))
        return [round(float(np.percentile(t, p)), 5) for p in (10, 50, 90)]

    per_call = {"fwd": percentiles(lambda: gpa.attn_fwd(q, k, v, w.causal, w.scale), args.steps)}
    for m in gpa.MODES:
        per_call["bwd_" + m] = percentiles(
            lambda: gpa.attn_bwd(q, k, v, o, lse, u, m, w.causal, w.scale, workspace=ws[m]),
            args.steps)

    # Context: the paper's grouped-query capture layout (16 query heads sharing
    # 4 key/value heads, same N, d and input recipe), forward and backward alone.
    gqa = None
    if not args.no_gqa and w.name == "h16_n4096_d64":
        wg = S.WORKLOADS[6]
        xg = S.make_inputs(wg, 6000)
        qg, kg, vg, ug = (to_dev(xg[n]) for n in ("q", "k", "v", "do"))
        og, lg = gpa.attn_fwd(qg, kg, vg, wg.causal, wg.scale)
        for _ in range(max(1, args.warmup // 2)):
            gpa.attn_fwd(qg, kg, vg, wg.causal, wg.scale)
        gqa = {"workload": wg.name, "Hq": wg.H, "Hkv": wg.kv_heads,
               "fwd_ms": round(timed(lambda: gpa.attn_fwd(qg, kg, vg, wg.causal, wg.scale),
                                     args.steps), 5), "bwd_ms": {}}
        # The modes are timed in interleaved rounds and each keeps its fastest
        # round: timed one after the other, the first mode would fall in the
        # clock transient that follows the preceding sections.
        fns = {}
        for m in gpa.MODES:
            wsg = torch.empty(gpa.attn_bwd_workspace_bytes(wg.B, wg.H, wg.N, wg.d, m, wg.kv_heads),
                              dtype=torch.uint8, device=dev)
            fns[m] = (lambda m_, w_: lambda: gpa.attn_bwd(qg, kg, vg, og, lg, ug, m_, wg.causal,
                                                          wg.scale, workspace=w_))(m, wsg)
        for _ in range(3):
            for m in gpa.MODES:
                fns[m]()
                t = round(timed(fns[m], args.steps), 5)
                gqa["bwd_ms"][m] = min(gqa["bwd_ms"].get(m, t), t)
        gpa.profile_enable(True)
        for _ in range(args.steps):
            fns["gproj"]()
        torch.cuda.synchronize()
        gprof = gpa.profile_read()
        gpa.profile_enable(False)
        gqa["kernels_ms"] = {n: round(t / c, 5) for n, (t, c) in gprof.items() if c}
        gqa["gproj_bwd_overhead_vs_plain_pct"] = round(
            100.0 * (gqa["bwd_ms"]["gproj"] / gqa["bwd_ms"]["plain"] - 1), 2)
        del qg, kg, vg, ug, og, lg

    # The fused FP32 attention (forward + backward in one call, BF16 I/O, FP32
    # products and accumulation on the FP32 matrix cores): the accuracy-class
    # baseline, timed beside the BF16 path, with its own fraction of the FP32
    # peak by the standard count and per kernel.
    for _ in range(2):
        gpa.fp32_attn(q, k, v, u, w.causal, w.scale)
    fp32_ms = timed(lambda: gpa.fp32_attn(q, k, v, u, w.causal, w.scale), max(5, args.steps // 5))
    gpa.profile_enable(True)
    for _ in range(max(5, args.steps // 5)):
        gpa.fp32_attn(q, k, v, u, w.causal, w.scale)
    torch.cuda.synchronize()
    fprof = gpa.profile_read()
    gpa.profile_enable(False)
    fp32_kern = {n: round(t / c, 5) for n, (t, c) in fprof.items() if c and n.startswith("fp32")}
    fp32 = {"fwd_bwd_ms": round(fp32_ms, 5),
            "tflops_standard_count": round(flops / (fp32_ms * 1e-3) / 1e12, 2),
            "frac_of_fp32_peak": round(flops / (fp32_ms * 1e-3) / 1e12 / PEAK_FP32_TFLOPS, 4),
            "peak": PEAK_FP32_TFLOPS, "kernels_ms": fp32_kern,
            # products per causal pair each kernel executes (fwd QK^T, PV; query
            # pass QK^T, dO V^T, dS K; key pass QK^T, dO V^T, P^T dO, dS^T Q)
            "kernel_frac_executed": {
                n: round(p * 2.0 * d * B * H * N * N / 2.0 / (fp32_kern[n] * 1e-3) / 1e12
                         / PEAK_FP32_TFLOPS, 4)
                for n, p in (("fp32_fwd", 2), ("fp32_dq", 3), ("fp32_dkdv", 4)) if n in fp32_kern}}

    # Roofline of the dominant kernel.  Algorithmic flops count each dense
    # contraction of the method once over the whole path (forward: QK^T, PV;
    # backward: QK^T, dO V^T, tK, r^T dO, t^T Q, and for GProj rK and r^T z):
    # a kernel is credited only with the products it forms first.  The key pass
    # recomputes S = QK^T and dP = dO V^T, which the query pass already formed
    # (schedule-dependent recompute, reported separately as executed products).
    pairs = B * H * N * N / 2.0
    flop_pair = 2.0 * d  # one dense contraction per causal (query, key) pair
    dom = max((n for n in kern if n in ALG_PRODUCTS), key=lambda n: kern[n])
    alg_p = ALG_PRODUCTS[dom][args.mode]
    exe_p = EXEC_PRODUCTS[dom][args.mode]
    alg = alg_p * flop_pair * pairs
    achieved = alg / (kern[dom] * 1e-3) / 1e12
    bwd_kern_ms = sum(kern[n] for n in ("bwd_dq", "bwd_dkdv") if n in kern)
    bwd_alg_products = {"plain": 5, "gproj_q": 6, "gproj": 7}[args.mode]
    roofline = {"kernel": dom, "bound": "mfma", "achieved": round(achieved, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": recorded_traffic(dom, args.mode, w.name),
                "avg_ms": round(kern[dom], 5),
                "algorithmic_products_per_pair": alg_p,
                "algorithmic_flops_per_launch": alg,
                "executed_products_per_pair": exe_p,
                "executed_frac": round(exe_p * flop_pair * pairs / (kern[dom] * 1e-3) / 1e12
                                       / PEAK_BF16_TFLOPS, 4),
                # the whole backward of this mode (both passes) by the method's
                # algorithmic count: plain 5, gproj_q 6, gproj 7 products per pair
                "backward_algorithmic_products_per_pair": bwd_alg_products,
                "backward_kernels_ms": round(bwd_kern_ms, 5),
                "backward_frac": round(bwd_alg_products * flop_pair * pairs / (bwd_kern_ms * 1e-3)
                                       / 1e12 / PEAK_BF16_TFLOPS, 4)}
    # The nominal peak assumes 2.4 GHz; the part sustains less under this load.
    # The clock the dominant kernel ran at in the committed counter pass (null
    # when the record is stale) gives the peak at that clock.
    clk = recorded_clock(dom, args.mode, w.name)
    roofline["sustained_clock_ghz"] = clk
    roofline["peak_at_sustained_clock"] = (None if clk is None
                                           else round(PEAK_BF16_TFLOPS * clk / NOMINAL_CLOCK_GHZ, 1))
    roofline["frac_at_sustained_clock"] = (None if clk is None
                                           else round(achieved / roofline["peak_at_sustained_clock"], 4))

    best_plain = min(("plain", "plain_atomic_dq"), key=lambda m: bwd_ms[m])
    out = {
        "metric": METRIC, "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": B, "H": H, "N": N, "d": d, "causal": True,
                   "mode": args.mode, "scale": w.scale, "k_bias_std": w.k_bias_std,
                   "do_std": w.do_std, "seed": seed},
        "roofline": roofline,
        "kernels_ms": {k2: round(v2, 5) for k2, v2 in kern.items()},
        "fwd_ms": round(fwd_ms, 5),
        "bwd_ms": {m: round(t, 5) for m, t in bwd_ms.items()},
        "per_call_ms_p10_p50_p90": per_call,
        # overheads against the fastest plain backward measured here (the
        # two-pass schedule or the single pass with atomic dQ)
        "best_plain": best_plain,
        "plain_atomic_dq_kernels_ms": atomic_kern["plain"],
        "atomic_schedule_kernels_ms": {m: atomic_kern[m] for m in ("gproj_q", "gproj")},
        "gproj_bwd_overhead_vs_plain_pct": round(100.0 * (bwd_ms["gproj"] / bwd_ms[best_plain] - 1), 2),
        "gproj_q_bwd_overhead_vs_plain_pct": round(100.0 * (bwd_ms["gproj_q"] / bwd_ms[best_plain] - 1), 2),
        "fp32_attn": fp32,
        "fp32_attn_vs_gproj_fwd_bwd": round(fp32_ms / (fwd_ms + bwd_ms["gproj"]), 3),
        "wall_s_timed": round(wall, 3),
        "ms_per_step_steady_after_200_more_steps": round(ms_steady, 5),
    }
    if gqa is not None:
        out["gqa"] = gqa

    # The memory-bound kernels against the HBM roofline: compulsory bytes per
    # launch over the kernel's measured duration.  The group sum of the
    # grouped-query backward, and the atomic schedule's preprocess and finalize
    # kernels (the two-pass schedule folds those steps into its passes).
    hbm = {}

    def hbm_entry(name, ms_k, nbytes, what):
        gbs = nbytes / (ms_k * 1e-3) / 1e9
        kname, kmode = name.rsplit("/", 1)
        hbm[name] = {"ms": round(ms_k, 5), "bytes": int(nbytes), "achieved_GB_s": round(gbs, 1),
                     "peak_GB_s": PEAK_HBM_GBS, "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "bytes_counted": what,
                     # calibrated FETCH_SIZE + WRITE_SIZE of the committed PMC summary
                     "traffic": recorded_traffic(kname, kmode)}

    ten = B * H * N * d                      # elements of one [B, H, N, d] tensor
    rows = B * H * N
    tile_stats = B * H * ((N + 63) // 64) * 128 * 4
    ak = atomic_kern
    hbm_entry("bwd_pre/plain", ak["plain"]["bwd_pre"], 2 * ten * 2 + rows * 4 + tile_stats + ten * 4,
              "read O, dO, LSE; write the tile statistics; zero A")
    hbm_entry("bwd_pre/gproj", ak["gproj"]["bwd_pre"],
              2 * ten * 2 + rows * 4 + tile_stats + 2 * ten * 4 + 2 * rows * 4,
              "read O, dO, LSE; write the tile statistics; zero A, B, rho, m")
    hbm_entry("bwd_dq_finalize/plain", ak["plain"]["bwd_dq_finalize"], ten * 4 + ten * 2,
              "read A; write dQ")
    hbm_entry("bwd_gproj_finalize/gproj", ak["gproj"]["bwd_dq_finalize"],
              2 * ten * 4 + 2 * rows * 4 + ten * 2 + 2 * ten * 2,
              "read A, B, rho, m, Q; write dQ, -z")
    if gqa is not None and "group_sum" in gqa.get("kernels_ms", {}):
        wg = S.WORKLOADS[6]
        hbm_entry("group_sum/" + wg.name + "/gproj", gqa["kernels_ms"]["group_sum"],
                  2 * wg.B * wg.H * wg.N * wg.d * 4 + 2 * wg.B * wg.kv_heads * wg.N * wg.d * 2,
                  "read the FP32 dK, dV contributions of every query head; write BF16 dK, dV")
    out["hbm_bound_kernels"] = hbm

    # The wider-head, long-sequence and batched workloads, timed on the same
    # kernels (their parity is covered by the tests): forward and backward per
    # mode, the GProj overhead and each kernel's fraction of the bf16 peak by
    # its algorithmic products.
    if not args.no_configs and w.name == "h16_n4096_d64":
        out["configs"] = {}
        orc = None
        if not args.no_accuracy:
            import oracle as orc
        # at least 50 calls or 200 ms of each: 50, 50, 10 calls
        for idx, iters in ((3, 50), (4, 50), (5, 10)):
            wc = S.WORKLOADS[idx]
            out["configs"][wc.name] = time_config(
                gpa, S, wc, 1000 * idx, iters, dev, to_dev,
                oracle=orc,
                heads=None if idx == 3 else ([(0, 0), (0, 15)] if idx == 4 else [(0, 0), (7, 31)]))

    if not args.no_accuracy or not args.no_cpu_baseline:
        import oracle
        # A bounded sample: whole heads, as many as fit ~20 s of the oracle
        # (the reference workload takes ~1 s whole on 16 host threads).
        per_head_s = 1.0 / 16 * (N / 4096) ** 2 * (d / 64)
        nh = min(B * H, max(1, int(20.0 / per_head_s)))
        flat = lambda a: a.reshape(B * H, N, -1)[:nh]  # noqa: E731
        xs = {n: flat(x[n]) for n in ("q", "k", "v", "do")}
        t0 = time.perf_counter()
        ex = oracle.exact(xs["q"], xs["k"], xs["v"], xs["do"], w.causal, w.scale)
        cpu_s = time.perf_counter() - t0
        scope = (f"whole workload ({B * H} heads" if nh == B * H
                 else f"{nh} of {B * H} heads (")
        if not args.no_cpu_baseline:
            # When the sample takes well under 10 s, run it again until about
            # 10 s of oracle time have passed, and report the mean.
            runs = [cpu_s]
            while sum(runs) < 10.0 and len(runs) < 64:
                t0 = time.perf_counter()
                oracle.exact(xs["q"], xs["k"], xs["v"], xs["do"], w.causal, w.scale)
                runs.append(time.perf_counter() - t0)
            mean_s = sum(runs) / len(runs)
            out["cpu_baseline"] = {"value": round(flops * nh / (B * H) / mean_s / 1e12, 6),
                                   "unit": "TFLOP/s", "cores": oracle.max_threads(),
                                   "kind": "oracle",
                                   "sample": f"{scope}, N={N}, d={d}): exact FP64 forward + VJP, "
                                             f"C/OpenMP, {len(runs)} runs, {sum(runs):.1f} s, "
                                             f"mean {mean_s:.2f} s per run",
                                   "seconds": round(mean_s, 3), "runs": len(runs)}
        if not args.no_accuracy:
            acc = {}
            fo, flse, fdq, fdk, fdv = gpa.fp32_attn(q, k, v, u, w.causal, w.scale)
            res = {"fp32": (fo, fdq, fdk, fdv)}
            for m in gpa.MODES:
                dq, dk, dv = gpa.attn_bwd(q, k, v, o, lse, u, m, w.causal, w.scale, workspace=ws[m])
                res[m] = (o, dq, dk, dv)
            # FA3 as the paper describes it: the historical FMA exponent rounding
            # in the forward, then the plain backward on its O and LSE.
            of, lf = gpa.attn_fwd_fma(q, k, v, w.causal, w.scale)
            res["fa3_fma_plain"] = (of, *gpa.attn_bwd(q, k, v, of, lf, u, "plain", w.causal,
                                                       w.scale, workspace=ws["plain"]))
            torch.cuda.synchronize()
            host = lambda t: t.reshape(B * H, N, -1)[:nh].float().cpu().numpy().astype(np.float64)  # noqa: E731
            for m, (oo, dq, dk, dv) in res.items():
                acc[m] = {n: round(oracle.rel_l2(host(t), ex[n]), 4)
                          for n, t in (("O", oo), ("dQ", dq), ("dK", dk), ("dV", dv))}
            out["rel_l2_pct_vs_fp64"] = acc
            if not args.no_seeds and nh == B * H:
                out["seed_protocol"] = seed_protocol(gpa, S, oracle, w, wid[w.name], to_dev)
            # Context: the regime of the paper's captures (near one-hot rows at
            # a logit scale of ~10^4, large common key offset), where the
            # forward's exponent rounding matters: FA3 (FMA forward + plain),
            # FA3-SBS (plain) and GProj, N = 1024, two heads.
            ws_ = S.Workload("sharp regime", 1, 2, 1024, 64, q_std=3000.0, k_bias_std=64.0,
                             do_std=1.0)
            xs_ = S.make_inputs(ws_, 777)
            qs_, ks_, vs_, us_ = (to_dev(xs_[n]) for n in ("q", "k", "v", "do"))
            exs_ = oracle.exact(xs_["q"], xs_["k"], xs_["v"], xs_["do"], True, ws_.scale)
            sharp = {}
            for name, fwd, m in (("fa3_fma_plain", gpa.attn_fwd_fma, "plain"),
                                 ("plain", gpa.attn_fwd, "plain"), ("gproj", gpa.attn_fwd, "gproj")):
                oo, ll = fwd(qs_, ks_, vs_, True, ws_.scale)
                dq, dk, dv = gpa.attn_bwd(qs_, ks_, vs_, oo, ll, us_, m, True, ws_.scale)
                torch.cuda.synchronize()
                hs = lambda t: t.float().cpu().numpy().astype(np.float64)  # noqa: E731
                sharp[name] = {n: round(oracle.rel_l2(hs(t), exs_[n]), 4)
                               for n, t in (("O", oo), ("dQ", dq), ("dK", dk), ("dV", dv))}
            fo, _, fdq, fdk, fdv = gpa.fp32_attn(qs_, ks_, vs_, us_, True, ws_.scale)
            torch.cuda.synchronize()
            sharp["fp32"] = {n: round(oracle.rel_l2(hs(t), exs_[n]), 4)
                             for n, t in (("O", fo), ("dQ", fdq), ("dK", fdk), ("dV", fdv))}
            out["rel_l2_pct_sharp_regime"] = {"workload": "q_std 3000, k_bias_std 64, 2 heads, "
                                                          "N 1024, d 64, causal", **sharp}
    if args.calibrate_copy:
        # A plain device copy of known size: FETCH_SIZE / WRITE_SIZE of this
        # kernel calibrate the counters of the attention kernels.  The source
        # is evicted from the 256 MiB last-level cache first (a 512 MiB fill of
        # another buffer), so the copy reads it from HBM.
        n = 128 * 1024 * 1024  # int32 elements: 512 MiB
        a = torch.ones(n, dtype=torch.int32, device=dev)
        flush = torch.empty(n, dtype=torch.int32, device=dev)
        b = torch.empty_like(a)
        flush.fill_(3)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        out["calibration_copy_bytes"] = n * 4
        del a, b, flush
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
