#!/usr/bin/env python3
"""Benchmark of the chunked MoE expert layer on one MI355X.

One step = one pass of the whole hot path over one batch of received tokens:
expert counts (the paper's "first notification") -> memory-aware chunk plan
(Eq. (8)/(9) + bins) -> chunked forward (Eq. (6)) -> chunked-recompute
backward (Eq. (7)).  Inputs are synthetic, seeded, and resident in HBM before
the timed region starts.

The default workload is the largest single-GPU one: the paper's per-GPU
worst case of e*s*t_k = 32*4096*8 = 1 048 576 token-slots (131072 received
tokens x top-8, h = 7168, F = 2048, 32 local experts, one expert taking half
of the slots), with the chunk count the planner picks for an 8 GB activation
budget.

Prints ONE JSON line (rank 0, N = 1 GPU):
  value        received tokens per second (whole job = one GPU)
  roofline     the dominant kernel against its roofline (algorithmic flops
               or bytes per launch over its mean launch time, HIP events on
               the launch stream inside the timed region)
  gemm         every grouped GEMM's algorithmic TFLOP/s and share of the
               bf16 peak, beside the 60 % target
  gemm_reference  the vendor library's batched bf16 GEMM at FC1's shape
               (uniform rows per expert, no gather) beside FC1's own rate
  clock        the graphics clock through the timed steps (amdsmi), and the
               layer's executed flops against the peak scaled to it
  hbm_kernels  the memory-bound steps' algorithmic GB/s against 8 TB/s and
               against a plain streaming copy measured in the same run
               (hbm_copy_reference)
  cpu_baseline the fp64 oracle on the host cores, on a bounded token sample
  chunks_sweep tokens/s and measured peak activation bytes for every chunk
               count of the workload, beside the memory-model predictions
  budget_sweep the planner's chunk count per activation budget with the
               measured peak (workload 5: 4-64 GB; the dense-FFN workload 3,
               where the backward holds more per slot than Table 2's rows)
  chunk_order  the same step with expert-ordered chunks (a variant outside
               the paper: runs of whole experts per chunk) beside the
               paper's token-range chunks, on this workload and workload 4
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
PEAK_HBM_GBS = 8000.0

# activation budget handed to the planner per workload (bytes); the plan
# then picks C from the bins
DEFAULT_BUDGET = {1: 64 * 1024, 2: 250 * 10**6, 3: 500 * 10**6, 4: 10**9, 5: 8 * 10**9}
# activation budgets swept through the planner (workload 5: 4 GB to 64 GB);
# each budget's C is joined with the measured chunk sweep
BUDGET_SWEEP = {5: [4 * 10**9, 8 * 10**9, 16 * 10**9, 32 * 10**9, 64 * 10**9],
                3: [5 * 10**8, 10**9, 13 * 10**8, 2 * 10**9, 25 * 10**8, 4 * 10**9]}
# router logits per token: the 32 local experts of workloads 4 and 5 are one
# GPU's slice of a 256-expert model (the paper's Table 3 models)
ROUTER_WIDTH = {4: 256, 5: 256}
GEMMS = ("fc1", "fc2", "fc1_recompute", "fc2_dgrad", "fc2_wgrad", "fc1_wgrad", "fc1_dgrad")
GEMM_TARGET = 0.60   # share of the bf16 MFMA peak the grouped GEMMs aim for
HBM_KERNELS = ("combine", "unpermute")  # the memory-bound steps


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=5, help="workload number (1-5)")
    ap.add_argument("--budget", type=float, default=None, help="activation budget, bytes")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-router", action="store_true",
                    help="skip the router and block measurement")
    ap.add_argument("--no-budget3", action="store_true",
                    help="skip the workload-3 activation-budget sweep")
    ap.add_argument("--no-order", action="store_true",
                    help="skip the chunk-order comparison")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target duration of the oracle sample")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one plain 1 GiB device copy first (reference for HBM counters)")
    ap.add_argument("--summarize-traffic", metavar="DIR", default=None,
                    help="no GPU work: turn the FETCH_SIZE / WRITE_SIZE counter CSVs of two "
                         "rocprofv3 --pmc runs in DIR into profiles/fc1_wgrad_cfg<N>_traffic.json")
    ap.add_argument("--summarize-counters", metavar="CSV", default=None,
                    help="no GPU work: print, per grouped-GEMM kernel, the mean of every "
                         "counter in a rocprofv3 --pmc CSV per dispatch")
    ap.add_argument("--summarize-mfma", metavar="CSV", default=None,
                    help="no GPU work: print a per-kernel MFMA utilisation table from a "
                         "rocprofv3 --pmc CSV of SQ_VALU_MFMA_BUSY_CYCLES, "
                         "SQ_INSTS_VALU_MFMA_MOPS_BF16, GRBM_GUI_ACTIVE")
    return ap.parse_args()


def source_digest(kernel_file: str) -> str:
    path = os.path.join(ROOT, "paper_2511_21431_amd", "csrc", kernel_file)
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def read_traffic(kernel: str, workload: str):
    """HBM bytes per launch measured with rocprofv3 counters, if a summary for
    this kernel and workload exists and the kernel source has not changed
    since (the summary records the source digest)."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            d = json.load(f)
        if d.get("source_sha256_16") != source_digest(d.get("source", "grouped_gemm.hip")):
            return None
        return float(d["bytes_per_launch"])
    except Exception:
        return None


# ---- counter summaries (host only) ----------------------------------------
# The FC1 weight-gradient launches of the split-tail grid (whole tiles of the
# 256 x 256, 8-wave configuration); the two dW modes are separate kernels.
FC1_WGRAD_KEY = ("grouped_gemm_split_kernel",
                 "ProbWgrad<unsigned short, memfine::(anonymous namespace)::Cfg<256, 256, 2, 4, 2, 128, 3>, true, ")


def _counter_rows(path):
    import csv
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def summarize_traffic(d, cfg, path=None):
    """HBM bytes per FC1 weight-gradient launch from two counter runs, each
    counter scaled by what it reads for the 1 GiB elementwise pass
    (`--calibrate-copy`, kernel neg) in the same process.  Writes the summary
    to `path` (default profiles/fc1_wgrad_cfg<cfg>_traffic.json) and returns
    it."""
    per = {}
    scale = {}
    for ctr, key in (("FETCH_SIZE", "fetch"), ("WRITE_SIZE", "write")):
        rows = _counter_rows(os.path.join(d, f"{ctr}_counter_collection.csv"))
        ref = [float(r["Counter_Value"]) for r in rows if "neg_kernel" in r["Kernel_Name"]]
        if len(ref) != 1:
            raise SystemExit(f"{ctr}: expected one calibration dispatch, found {len(ref)}")
        scale[key] = (1 << 30) / (ref[0] * 1024.0)      # counter in KiB
        scale[key + "_kb"] = ref[0]
        for r in rows:
            n = r["Kernel_Name"]
            if all(k in n for k in FC1_WGRAD_KEY):
                e = per.setdefault(n, {"launches": 0, "fetch_bytes": 0.0, "write_bytes": 0.0})
                if key == "fetch":
                    e["launches"] += 1
                e[key + "_bytes"] += float(r["Counter_Value"]) * 1024.0 * scale[key]
    if not per:
        raise SystemExit("no FC1 weight-gradient dispatches in the counter files")
    # mean over every profiled launch: the two dW modes (the first chunk
    # writes dW, the others accumulate) weighted as a step runs them
    n_all = sum(e["launches"] for e in per.values())
    fetch = sum(e["fetch_bytes"] for e in per.values()) / n_all
    write = sum(e["write_bytes"] for e in per.values()) / n_all
    for e in per.values():
        e["fetch_bytes"] /= e["launches"]
        e["write_bytes"] /= e["launches"]
    out = {"kernel": "fc1_wgrad", "rocprof_name": " + ".join(sorted(per)),
           "launches_profiled": sum(e["launches"] for e in per.values()), "per_kernel": per,
           "fetch_bytes_per_launch": fetch, "write_bytes_per_launch": write,
           "bytes_per_launch": fetch + write,
           "copy_reference": {"bytes_each_way": float(1 << 30), "fetch_kb": scale["fetch_kb"],
                              "write_kb": scale["write_kb"], "fetch_scale": scale["fetch"],
                              "write_scale": scale["write"]},
           "source": "grouped_gemm.hip", "source_sha256_16": source_digest("grouped_gemm.hip")}
    if path is None:
        path = os.path.join(ROOT, "profiles", f"fc1_wgrad_cfg{cfg}_traffic.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(f"{path}: fetch {fetch:.4g} B + write {write:.4g} B per launch")
    for n, e in sorted(per.items()):
        print(f"  {n[-12:]}: {e['launches']} launches, fetch {e['fetch_bytes']:.4g}, "
              f"write {e['write_bytes']:.4g}")
    return out


def _gemm_dispatches(path):
    """Dispatches of the 256 x 256 grouped GEMMs in a counter CSV, keyed by
    the kernel's role; each with its duration (ns) and its counters."""
    import re
    rows = _counter_rows(path)
    disp = {}
    for r in rows:
        e = disp.setdefault(r["Dispatch_Id"], {"name": r["Kernel_Name"], "ns":
                            int(r["End_Timestamp"]) - int(r["Start_Timestamp"]), "ctr": {}})
        e["ctr"][r["Counter_Name"]] = e["ctr"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    out = {}
    for e in disp.values():
        m = re.search(r"(Prob\w+)<unsigned short, [^<]*Cfg<256, 256[^>]*>(?:, (true|false))?(?:, (\d))?",
                      e["name"])
        if not m or "split" not in e["name"]:
            continue
        k = {"ProbFC1": "fc1_recompute" if m.group(2) == "true" else "fc1", "ProbFC2": "fc2",
             "ProbFC2Dgrad": "fc2_dgrad", "ProbFC1Dgrad": "fc1_dgrad",
             "ProbWgrad": ("fc1_wgrad" if m.group(2) == "true" else "fc2_wgrad")
             + (", dW accumulated" if m.group(3) == "1" else ", dW written")}[m.group(1)]
        out.setdefault(k, []).append(e)
    return out


def summarize_counters(path):
    """Per grouped-GEMM kernel: launches, mean duration and the mean of each
    counter per dispatch (summed over the counter's instances)."""
    by = _gemm_dispatches(path)
    names = sorted({c for es in by.values() for e in es for c in e["ctr"]})
    print("| kernel | launches | avg us | " + " | ".join(names) + " |")
    print("|---|---:|---:|" + "---:|" * len(names))
    res = {}
    for k, es in sorted(by.items(), key=lambda kv: -sum(e["ns"] for e in kv[1])):
        n = len(es)
        mean = {c: sum(e["ctr"].get(c, 0.0) for e in es) / n for c in names}
        res[k] = {"launches": n, "avg_ns": sum(e["ns"] for e in es) / n, **mean}
        print(f"| {k} | {n} | {res[k]['avg_ns'] / 1e3:.1f} | "
              + " | ".join(f"{mean[c]:.4g}" for c in names) + " |")
    return res


def summarize_mfma(path):
    """Per GEMM kernel: MFMA busy share (rocprofv3's MfmaUtil: busy cycles
    summed over the SIMDs / (GUI-active cycles of one XCD x 1024 SIMDs); the
    CSV's GRBM_GUI_ACTIVE is the sum over the 8 XCDs) and the bf16 MFMA
    flops the matrix cores executed (MOPS x 512) against the dispatch time."""
    import re
    rows = _counter_rows(path)
    disp = {}
    for r in rows:
        e = disp.setdefault(r["Dispatch_Id"], {"name": r["Kernel_Name"], "ns":
                            int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
        e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    agg = {}
    for e in disp.values():
        m = re.search(r"(Prob\w+)<unsigned short, [^<]*Cfg<256, 256[^>]*>(?:, (true|false))?(?:, (\d))?",
                      e["name"])
        if not m or "split" not in e["name"]:
            continue
        k = {"ProbFC1": "fc1_recompute" if m.group(2) == "true" else "fc1", "ProbFC2": "fc2",
             "ProbFC2Dgrad": "fc2_dgrad", "ProbFC1Dgrad": "fc1_dgrad",
             "ProbWgrad": ("fc1_wgrad" if m.group(2) == "true" else "fc2_wgrad")
             + (", dW accumulated" if m.group(3) == "1" else ", dW written")}[m.group(1)]
        a = agg.setdefault(k, {"n": 0, "ns": 0, "busy": 0.0, "gui": 0.0, "mops": 0.0})
        a["n"] += 1
        a["ns"] += e["ns"]
        a["busy"] += e.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        a["gui"] += e.get("GRBM_GUI_ACTIVE", 0.0)
        a["mops"] += e.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
    print("| kernel | launches | avg us | MFMA busy (MfmaUtil) | executed bf16 TFLOP/s | of 2.5 PFLOP/s |")
    print("|---|---:|---:|---:|---:|---:|")
    for k, a in sorted(agg.items(), key=lambda kv: -kv[1]["ns"]):
        a["util"] = a["busy"] / (a["gui"] / 8.0 * 1024.0)
        a["tflops"] = a["mops"] * 512.0 / (a["ns"] * 1e-9) / 1e12
        print(f"| {k} | {a['n']} | {a['ns'] / a['n'] / 1e3:.1f} | {a['util'] * 100:.1f} % | "
              f"{a['tflops']:.0f} | {a['tflops'] / PEAK_TFLOPS['bf16'] * 100:.1f} % |")
    return agg


def main():
    args = parse()
    if args.summarize_traffic:
        summarize_traffic(args.summarize_traffic, args.config)
        return
    if args.summarize_mfma:
        summarize_mfma(args.summarize_mfma)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(the expert-parallel exchange between GPUs is not implemented), so --gpus "
              "must be 1", file=sys.stderr)
        sys.exit(2)

    import torch

    import moe_workloads as mw
    import paper_2511_21431_amd as mf

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    mf.lib()

    cfg = args.config
    w = mw.WORKLOADS[cfg]
    seed = cfg if args.seed is None else args.seed
    budget = int(args.budget) if args.budget is not None else DEFAULT_BUDGET[cfg]
    bins = w.bins
    dtype = mf.BF16 if w.dtype == "bf16" else mf.F32
    shape = mf.make_shape(w.T, w.h, w.F, w.E, w.k, dtype)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32

    log(f"[bench] workload {cfg} {w.name}: T={w.T} h={w.h} F={w.F} E={w.E} k={w.k} {w.dtype}")
    idx_np, gates_np = mw.make_routing(w, seed)
    dev = mw.make_tensors_device(w, seed, "cuda")
    idx = torch.from_numpy(idx_np).cuda()
    gates = torch.from_numpy(gates_np).cuda()
    Y = torch.empty((w.T, w.h), dtype=dt, device="cuda")
    dX = torch.empty_like(Y)
    dW1 = torch.empty((w.E, 2 * w.F, w.h), dtype=torch.float32, device="cuda")
    dW2 = torch.empty((w.E, w.h, w.F), dtype=torch.float32, device="cuda")
    dg = torch.empty((w.T, w.k), dtype=torch.float32, device="cuda")
    work = torch.zeros(w.E + 1, dtype=torch.int32, device="cuda")
    if args.calibrate_copy:
        # an elementwise pass over 1 GiB (reads 1 GiB, writes 1 GiB) whose
        # kernel name (neg) is unique in this process
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        del src, dst
    torch.cuda.synchronize()

    def step(C_fixed=None, allocator=None):
        counts = mf.memfine_count(shape, idx, work)            # syncs once
        rc, C, info = mf.memfine_plan(shape, counts, budget, bins=bins)
        if C_fixed is not None:
            C = C_fixed
        mf.memfine_moe_fwd(shape, C, dev["X"], idx, gates, dev["W1"], dev["W2"], Y,
                           allocator=allocator)
        mf.memfine_moe_bwd(shape, C, dev["X"], idx, gates, dev["W1"], dev["W2"], dev["dY"], dX,
                           dW1, dW2, dg, allocator=allocator)
        return C, info

    # ---- warm-up, and one fully instrumented step to find the dominant kernel
    for _ in range(max(args.warmup, 1)):
        C, plan_info = step()
    torch.cuda.synchronize()
    mf.memfine_profile_begin()
    step()
    torch.cuda.synchronize()
    prof_all = mf.memfine_profile_end()
    dominant = max(prof_all, key=lambda k: prof_all[k]["total_ms"])
    log(f"[bench] plan: C={C} (c_theory={plan_info['c_theory']}, s''={plan_info['s_recv']}, "
        f"budget={budget}); dominant kernel: {dominant}")
    for k, v in sorted(prof_all.items(), key=lambda kv: -kv[1]["total_ms"]):
        log(f"[bench]   {k:14s} {v['launches']:3d} launches {v['total_ms']:8.3f} ms "
            f"{v['flops'] / max(v['total_ms'], 1e-9) / 1e9:8.1f} TFLOP/s "
            f"{v['bytes'] / max(v['total_ms'], 1e-9) / 1e6:8.1f} GB/s")

    # ---- timed region
    mf.memfine_profile_begin([dominant])
    torch.cuda.synchronize()
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    with ClockSampler() as clock:
        t0 = time.perf_counter()
        ends[0].record()
        for i in range(args.steps):
            step()
            ends[i + 1].record()   # per-step GPU time between consecutive step ends
        torch.cuda.synchronize()
        t1 = time.perf_counter()
    clock = clock.summary()
    prof = mf.memfine_profile_end()
    step_ms = sorted(a.elapsed_time(b) for a, b in zip(ends, ends[1:]))
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    tokens_per_s = w.T * args.steps / (t1 - t0)
    d = prof[dominant]
    avg_ms = d["total_ms"] / d["launches"]
    flops_per_launch = d["flops"] / d["launches"]
    bytes_per_launch = d["bytes"] / d["launches"]
    peak = PEAK_TFLOPS[w.dtype]
    # the kernel's roofline: whichever of its algorithmic flops at the MFMA
    # peak and its algorithmic bytes at the HBM peak takes longer
    t_mfma = flops_per_launch / (peak * 1e12)
    t_hbm = bytes_per_launch / (PEAK_HBM_GBS * 1e9)
    bound = "hbm" if t_hbm > t_mfma else "mfma"
    achieved_tflops = flops_per_launch / (avg_ms * 1e-3) / 1e12
    achieved_gbs = bytes_per_launch / (avg_ms * 1e-3) / 1e9
    achieved = achieved_gbs if bound == "hbm" else achieved_tflops
    traffic = read_traffic(dominant, f"cfg{cfg}")
    executed_flops = 22.0 * w.N * w.h * w.F
    if clock:
        log(f"[bench] clock during the timed steps: mean {clock['mean_ghz']:.2f} GHz "
            f"(min {clock['min_ghz']:.2f}, max {clock['max_ghz']:.2f}, {clock['samples']} samples)")
    log(f"[bench] {ms_per_step:.3f} ms/step, {tokens_per_s:.0f} tokens/s, dominant {dominant} "
        f"avg {avg_ms:.3f} ms {achieved_tflops:.1f} TFLOP/s {achieved_gbs:.1f} GB/s ({bound}-bound)")

    # ---- what a plain streaming copy reaches on this part: the reference for
    # the memory-bound kernels besides the 8 TB/s nameplate
    copy_ref = hbm_copy_reference(torch)
    hbm_kernels = {}
    for k in HBM_KERNELS:
        v = prof_all.get(k)
        if v and v["total_ms"] > 0:
            gbs = v["bytes"] / (v["total_ms"] * 1e-3) / 1e9
            hbm_kernels[k] = {"ms": round(v["total_ms"], 4), "gbs": round(gbs, 1),
                              "frac_of_peak": round(gbs / PEAK_HBM_GBS, 4),
                              "frac_of_copy": round(gbs / copy_ref["gbs"], 4)}
    gemm_ref = None
    if w.dtype == "bf16":
        rows_ref = max(256, -(-w.T // C) * w.k // w.E)
        gemm_ref = gemm_reference(torch, w.E, rows_ref, 2 * w.F, w.h)
        fc1 = prof_all.get("fc1")
        if fc1 and fc1["total_ms"] > 0:
            gemm_ref["fc1_tflops"] = round(fc1["flops"] / (fc1["total_ms"] * 1e-3) / 1e12, 1)
            gemm_ref["fc1_frac_of_reference"] = round(gemm_ref["fc1_tflops"] / gemm_ref["tflops"], 4)
        log(f"[bench] vendor batched GEMM at FC1's shape ({w.E} x {rows_ref} rows): "
            f"{gemm_ref['tflops']:.0f} TFLOP/s; FC1 {gemm_ref.get('fc1_tflops')} TFLOP/s")
    log(f"[bench] streaming copy: {copy_ref['gbs']:.0f} GB/s; " +
        ", ".join(f"{k} {v['gbs']:.0f} GB/s ({v['frac_of_copy']:.2f} of it)"
                  for k, v in hbm_kernels.items()))

    # ---- chunk-count sweep: throughput and measured peak activation memory
    sweep = []
    if not args.no_sweep:
        for Cs in w.chunks:
            for _ in range(2):
                step(Cs)
            torch.cuda.synchronize()
            n_t = max(3, args.steps // 4)
            a = time.perf_counter()
            for _ in range(n_t):
                step(Cs)
            torch.cuda.synchronize()
            tps = w.T * n_t / (time.perf_counter() - a)
            alloc = mf.TorchAllocator()
            torch.cuda.synchronize()
            gc.collect()
            torch.cuda.reset_peak_memory_stats()
            base = torch.cuda.memory_allocated()
            step(Cs, allocator=alloc)
            torch.cuda.synchronize()
            peak_b = torch.cuda.max_memory_allocated() - base
            n_max = -(-w.T // Cs) * w.k
            beta_paper = (2 if w.dtype == "bf16" else 4) * (2 * w.h + 2 * w.F)
            sweep.append({
                "chunks": Cs, "tokens_per_s": round(tps, 1),
                "peak_activation_bytes": int(peak_b),
                "allocator_high_water_bytes": int(alloc.high_water),
                "predicted_bytes_impl": mf.memfine_workspace_bytes(shape, Cs, mf.PASS_BWD),
                "predicted_bytes_paper_model": beta_paper * n_max,
            })
            log(f"[bench] sweep C={Cs}: {tps:.0f} tokens/s, peak activation {peak_b / 1e9:.3f} GB")

    # ---- activation-budget sweep: the planner's C per budget (Eq. (8)/(9) +
    # bins from this workload's counts), with that C's measured throughput
    # and peak activation from the chunk sweep
    budget_sweep = None
    if cfg in BUDGET_SWEEP:
        counts = mf.memfine_count(shape, idx, work)
        by_c = {r["chunks"]: r for r in sweep}
        budget_sweep = []
        for b in BUDGET_SWEEP[cfg]:
            rc_b, C_b, info_b = mf.memfine_plan(shape, counts, b, bins=bins)
            r = by_c.get(C_b, {})
            budget_sweep.append({
                "budget_bytes": b, "status": mf.memfine_status_str(rc_b), "chunks": C_b,
                "c_theory": info_b["c_theory"], "paper_model_chunks": info_b["paper_chunks"],
                "tokens_per_s": r.get("tokens_per_s"),
                "peak_activation_bytes": r.get("peak_activation_bytes"),
                "predicted_bytes_impl": info_b["workspace_bytes"],
                "predicted_bytes_paper_model": r.get("predicted_bytes_paper_model"),
                "within_budget": (r["peak_activation_bytes"] <= b) if r else None})
            log(f"[bench] budget {b / 1e9:.0f} GB: C={C_b} (c={info_b['c_theory']}), "
                f"{r.get('tokens_per_s')} tokens/s, peak {r.get('peak_activation_bytes')} B")

    # ---- the same on the dense-FFN workload 3 (F > h: the backward holds
    # more bytes per slot than Table 2's rows), each budget's C run once with
    # the allocator hook
    budget_sweep3 = None
    if cfg != 3 and not args.no_budget3 and not args.no_sweep:
        budget_sweep3 = sweep_budgets(mf, torch, 3)

    # ---- MACT from the model configuration (Eq. (1)-(3), Section 4.2
    # thresholds) for the paper's Model I, beside the counts-based plan
    mact = mact_model_plan(mf, int(sum(mf.memfine_count(shape, idx, work))))

    # ---- expert-ordered chunks beside the paper's token-range chunks
    chunk_order = None
    if not args.no_order:
        chunk_order = {f"workload{cfg}": compare_orders(mf, torch, step, max(3, args.steps // 2),
                                                        w, peak)}
        if cfg != 4 and not args.no_sweep:
            chunk_order["workload4"] = compare_orders_workload(mf, torch, 4, max(3, args.steps // 2))

    # ---- the router in front of the layer: its kernels, and the whole block
    router = None
    if not args.no_router and w.k <= 16:
        router = bench_router(mf, torch, w, dev, step, args.steps, ROUTER_WIDTH.get(cfg, w.E))

    # ---- the oracle on the host cores, bounded sample of the same workload
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, idx_np, gates_np, dev, C, args.cpu_seconds)

    out = {
        "metric": "chunked MoE layer fwd+bwd tokens/sec on 1 GPU",
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded routing and N(0,1)/N(0,0.02) tensors)",
        "config": {"workload": f"{w.name}: T={w.T} received tokens, h={w.h}, F={w.F}, "
                               f"E={w.E} local experts, top-{w.k}",
                   "T": w.T, "h": w.h, "F": w.F, "E": w.E, "k": w.k,
                   "chunks": C, "budget_bytes": budget, "bins": list(bins),
                   "parallelism": "single GPU (one expert-parallel share)"},
        "step_ms_median": round(step_ms[len(step_ms) // 2], 4),
        "step_ms_min": round(step_ms[0], 4),
        "slots_per_s": round(w.N * args.steps / (t1 - t0), 1),
        # algorithmic (executed) flops of the step, 22 N h F, over the step
        # time, as a share of the bf16 peak: not a hardware MFMA counter
        "layer_flops_frac_of_peak": round(executed_flops / (ms_per_step * 1e-3) / 1e12 / peak, 4),
        "layer_tflops": round(executed_flops / (ms_per_step * 1e-3) / 1e12, 1),
        # the clock the chip held during the timed steps, and the layer's
        # executed flops against the bf16 peak scaled to that clock (the
        # 2.5 PFLOP/s figure assumes 2.4 GHz)
        "clock": clock,
        "layer_flops_frac_of_peak_at_clock": (
            round(executed_flops / (ms_per_step * 1e-3) / 1e12 / (peak * clock["mean_ghz"] / 2.4), 4)
            if clock else None),
        "gemm": gemm_table(prof_all, peak),
        "gemm_target_frac_of_peak": GEMM_TARGET,
        "roofline": {"kernel": dominant, "bound": bound, "achieved": round(achieved, 1),
                     "peak": PEAK_HBM_GBS if bound == "hbm" else peak,
                     "unit": "GB/s" if bound == "hbm" else "TFLOP/s",
                     "frac": round(achieved / (PEAK_HBM_GBS if bound == "hbm" else peak), 4),
                     "traffic": traffic, "avg_launch_ms": round(avg_ms, 4),
                     "launches": d["launches"], "flops_per_launch": flops_per_launch,
                     "bytes_per_launch": bytes_per_launch,
                     "achieved_tflops": round(achieved_tflops, 1),
                     "achieved_gbs": round(achieved_gbs, 1)},
        "kernels_one_step": {k: {"ms": round(v["total_ms"], 4),
                                 "tflops": round(v["flops"] / max(v["total_ms"], 1e-9) / 1e9, 1),
                                 "gbs": round(v["bytes"] / max(v["total_ms"], 1e-9) / 1e6, 1)}
                             for k, v in prof_all.items()},
        "layer_roofline_frac": round(layer_bound_ms(prof_all, peak) / ms_per_step, 4),
        "hbm_copy_reference": copy_ref,
        "gemm_reference": gemm_ref,
        "hbm_kernels": hbm_kernels,
        "chunks_sweep": sweep,
        "budget_sweep": budget_sweep,
        "budget_sweep_workload3": budget_sweep3,
        "mact_model_plan": mact,
        "chunk_order": chunk_order,
        "router": router,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


class ClockSampler:
    """The GPU's current graphics clock (amdsmi), sampled every `period`
    seconds by a daemon thread while the timed steps run.  Everything amdsmi
    does happens on that thread, so a failing or slow query never holds up
    the measurement; without amdsmi the summary is None.  So it is too when
    the timed steps take less than `min_seconds`: the reading does not follow
    short bursts (it stayed at 0.2 GHz through 0.3 s of full load)."""

    min_seconds = 2.0

    def __init__(self, period=0.01):
        import threading
        self.period, self.samples, self.seconds = period, [], 0.0
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        try:
            import amdsmi
            amdsmi.amdsmi_init()
        except Exception:
            return
        try:
            h = amdsmi.amdsmi_get_processor_handles()[0]
            while not self._stop.is_set():
                mhz = amdsmi.amdsmi_get_clock_info(h, amdsmi.AmdSmiClkType.GFX)["clk"]
                if isinstance(mhz, (int, float)):
                    self.samples.append(float(mhz))
                self._stop.wait(self.period)
        except Exception:
            pass
        finally:
            try:
                amdsmi.amdsmi_shut_down()
            except Exception:
                pass

    def __enter__(self):
        import time
        self._t0 = time.perf_counter()
        self._thread.start()
        return self

    def __exit__(self, *exc):
        import time
        self.seconds = time.perf_counter() - self._t0
        self._stop.set()
        self._thread.join(timeout=1.0)

    def summary(self):
        v = list(self.samples)
        if not v or self.seconds < self.min_seconds:
            return None
        return {"mean_ghz": round(sum(v) / len(v) / 1e3, 3), "min_ghz": round(min(v) / 1e3, 3),
                "max_ghz": round(max(v) / 1e3, 3), "samples": len(v),
                "source": "amdsmi current GFX clock every 10 ms during the timed steps"}


def gemm_reference(torch, E, rows, n, kdim, reps=5):
    """Best of `reps` vendor batched bf16 GEMMs (torch.bmm, contiguous
    operands) of E x [rows x kdim] @ [kdim x n]: FC1's shape with every
    expert given the same row count and no gather, the dense-library
    reference for the grouped GEMMs under this part's power limit."""
    a = torch.randn(E, rows, kdim, device="cuda").bfloat16()
    b = (torch.randn(E, kdim, n, device="cuda") * 0.02).bfloat16().contiguous()
    c = torch.bmm(a, b)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        c = torch.bmm(a, b)
        e1.record()
        e1.synchronize()
        times.append(e0.elapsed_time(e1))
    del a, b, c
    ms = min(times)
    tf = 2.0 * E * rows * n * kdim / (ms * 1e-3) / 1e12
    return {"tflops": round(tf, 1), "ms": round(ms, 4), "experts": E, "rows_per_expert": rows,
            "n": n, "k": kdim, "kernel": "torch.bmm bf16 (vendor BLAS), best of 5"}


def hbm_copy_reference(torch, nbytes=1 << 30, reps=5):
    """Best of `reps` device-to-device copies of `nbytes` (read + write, both
    far beyond the last-level cache), timed with events: the bandwidth a plain
    streaming kernel reaches on this part."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        e1.synchronize()
        times.append(e0.elapsed_time(e1))
    del src, dst
    ms = min(times)
    return {"gbs": round(2.0 * nbytes / (ms * 1e-3) / 1e9, 1), "bytes_moved": 2 * nbytes,
            "ms": round(ms, 4), "kernel": "torch copy_ of a 1 GiB fp32 tensor (best of 5)",
            "frac_of_peak": round(2.0 * nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}


def gemm_table(prof, peak_tflops):
    """Each grouped GEMM of one instrumented step: algorithmic TFLOP/s (HIP
    events around its launches) and its share of the bf16 peak."""
    out = {}
    for k in GEMMS:
        v = prof.get(k)
        if not v or v["total_ms"] <= 0:
            continue
        tf = v["flops"] / (v["total_ms"] * 1e-3) / 1e12
        out[k] = {"ms": round(v["total_ms"], 4), "tflops": round(tf, 1),
                  "frac_of_peak": round(tf / peak_tflops, 4)}
    return out


def sweep_budgets(mf, torch, cfg):
    """The planner's chunk count for each activation budget of BUDGET_SWEEP on
    workload `cfg`, and one layer step at that count with the allocator hook:
    the measured peak activation against the budget.  Also the bin that
    Table 2's bytes per slot alone would give and whether this layer's
    workspace would have fit it."""
    import moe_workloads as mw
    w = mw.WORKLOADS[cfg]
    shape = mf.make_shape(w.T, w.h, w.F, w.E, w.k, mf.BF16)
    log(f"[bench] budget sweep, workload {cfg} {w.name}: generating inputs")
    idx_np, gates_np = mw.make_routing(w, cfg)
    dev = mw.make_tensors_device(w, cfg, "cuda")
    idx = torch.from_numpy(idx_np).cuda()
    gates = torch.from_numpy(gates_np).cuda()
    Y = torch.empty((w.T, w.h), dtype=torch.bfloat16, device="cuda")
    dX = torch.empty_like(Y)
    dW1 = torch.empty((w.E, 2 * w.F, w.h), dtype=torch.float32, device="cuda")
    dW2 = torch.empty((w.E, w.h, w.F), dtype=torch.float32, device="cuda")
    dg = torch.empty((w.T, w.k), dtype=torch.float32, device="cuda")
    work = torch.zeros(w.E + 1, dtype=torch.int32, device="cuda")
    counts = mf.memfine_count(shape, idx, work)
    rows = []
    for b in BUDGET_SWEEP[cfg]:
        rc, C, info = mf.memfine_plan(shape, counts, b, bins=w.bins)
        alloc = mf.TorchAllocator()
        torch.cuda.synchronize()
        gc.collect()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        mf.memfine_moe_fwd(shape, C, dev["X"], idx, gates, dev["W1"], dev["W2"], Y, allocator=alloc)
        mf.memfine_moe_bwd(shape, C, dev["X"], idx, gates, dev["W1"], dev["W2"], dev["dY"], dX,
                           dW1, dW2, dg, allocator=alloc)
        torch.cuda.synchronize()
        peak_b = torch.cuda.max_memory_allocated() - base
        Cp = info["paper_chunks"]
        ws_paper = mf.memfine_workspace_bytes(shape, Cp, mf.PASS_BWD)
        rows.append({"budget_bytes": b, "status": mf.memfine_status_str(rc), "chunks": C,
                     "c_theory": info["c_theory"], "beta": info["beta"],
                     "predicted_bytes_impl": info["workspace_bytes"],
                     "peak_activation_bytes": int(peak_b),
                     "allocator_high_water_bytes": int(alloc.high_water),
                     "within_budget": bool(alloc.high_water <= b),
                     "paper_model_chunks": Cp, "paper_model_beta": info["beta_paper"],
                     "paper_model_chunks_workspace_bytes": ws_paper,
                     "paper_model_chunks_within_budget": bool(ws_paper <= b)})
        log(f"[bench] workload {cfg} budget {b / 1e9:.2f} GB: C={C} (paper model {Cp}), "
            f"peak {peak_b / 1e9:.3f} GB, within budget: {alloc.high_water <= b}")
    del dev, Y, dX, dW1, dW2
    torch.cuda.empty_cache()
    return {"workload": f"{w.name}: T={w.T}, h={w.h}, F={w.F}, E={w.E}, top-{w.k}", "rows": rows}


# Table 3's Model I on the paper's setup (Section 5): 64 GB GPUs, 43.0 GB of
# static memory (Table 4), p = 4 pipeline stages, full recomputation
MODEL_I = dict(b=1, s=4096, h=7168, a=128, h_d=128, k_a=128, e_n=256, g_e=2048, t=1, c=1,
               v=1, p=4, D_t=2, full_recompute=1)
MODEL_I_GPU = dict(M_gpu=64 * 10**9, alpha=(9, 10), M_sta=43 * 10**9)


def compare_orders(mf, torch, step, steps, w, peak):
    """The step timed in both chunk orders (launch option chunk_order), same
    inputs and planner: ms/step, tokens/s, and per-GEMM TFLOP/s from one
    instrumented step of each."""
    res = {}
    for name, order in (("tokens", mf.CHUNK_TOKENS), ("experts", mf.CHUNK_EXPERTS)):
        mf.memfine_set_launch_options(chunk_order=order)
        try:
            step()
            torch.cuda.synchronize()
            mf.memfine_profile_begin()
            C, _ = step()
            torch.cuda.synchronize()
            prof = mf.memfine_profile_end()
            a = time.perf_counter()
            for _ in range(steps):
                step()
            torch.cuda.synchronize()
            el = time.perf_counter() - a
        finally:
            mf.memfine_set_launch_options()
        res[name] = {"chunks": C, "ms_per_step": round(el * 1e3 / steps, 4),
                     "tokens_per_s": round(w.T * steps / el, 1),
                     "gemm": gemm_table(prof, peak),
                     "combine_ms": round(prof.get("combine", {}).get("total_ms", 0.0), 4),
                     "unpermute_ms": round(prof.get("unpermute", {}).get("total_ms", 0.0), 4)}
        log(f"[bench] chunk order {name}: C={C}, {res[name]['ms_per_step']:.3f} ms/step, "
            f"{res[name]['tokens_per_s']:.0f} tokens/s")
    return res


def compare_orders_workload(mf, torch, cfg, steps):
    """compare_orders on workload `cfg` with its own inputs and budget."""
    import moe_workloads as mw
    w = mw.WORKLOADS[cfg]
    log(f"[bench] chunk order, workload {cfg} {w.name}: generating inputs")
    shape = mf.make_shape(w.T, w.h, w.F, w.E, w.k, mf.BF16)
    idx_np, gates_np = mw.make_routing(w, cfg)
    dev = mw.make_tensors_device(w, cfg, "cuda")
    idx = torch.from_numpy(idx_np).cuda()
    gates = torch.from_numpy(gates_np).cuda()
    Y = torch.empty((w.T, w.h), dtype=torch.bfloat16, device="cuda")
    dX = torch.empty_like(Y)
    dW1 = torch.empty((w.E, 2 * w.F, w.h), dtype=torch.float32, device="cuda")
    dW2 = torch.empty((w.E, w.h, w.F), dtype=torch.float32, device="cuda")
    dg = torch.empty((w.T, w.k), dtype=torch.float32, device="cuda")
    work = torch.zeros(w.E + 1, dtype=torch.int32, device="cuda")

    def step():
        counts = mf.memfine_count(shape, idx, work)
        rc, C, info = mf.memfine_plan(shape, counts, DEFAULT_BUDGET[cfg], bins=w.bins)
        mf.memfine_moe_fwd(shape, C, dev["X"], idx, gates, dev["W1"], dev["W2"], Y)
        mf.memfine_moe_bwd(shape, C, dev["X"], idx, gates, dev["W1"], dev["W2"], dev["dY"], dX,
                           dW1, dW2, dg)
        return C, info

    res = compare_orders(mf, torch, step, steps, w, PEAK_TFLOPS[w.dtype])
    del dev, Y, dX, dW1, dW2
    torch.cuda.empty_cache()
    return res


def mact_model_plan(mf, s_recv):
    """MACT's threshold table for Model I at every pipeline rank and the bin
    it selects for this step's received slots (the library's host entry
    points, Eq. (1)-(3) and Section 4.2)."""
    bins = (1, 2, 4, 8, 16)
    m = mf.make_model(**MODEL_I)
    ranks = []
    for r in range(MODEL_I["p"]):
        th = mf.memfine_mact_thresholds(m, r, MODEL_I_GPU["M_gpu"], *MODEL_I_GPU["alpha"],
                                        MODEL_I_GPU["M_sta"], bins)
        rc, C = mf.memfine_mact_select(bins, th, s_recv)
        ranks.append({"r_pp": r, "thresholds": th, "chunks": C,
                      "status": mf.memfine_status_str(rc)})
    log(f"[bench] MACT Model I, s''={s_recv}: " + ", ".join(f"rank {x['r_pp']} C={x['chunks']}"
                                                           for x in ranks))
    return {"model": "Table 3 Model I (h=7168, g_e=2048, s=4096), 64 GB GPU, alpha=0.9, "
                     "M_sta=43.0 GB, p=4, full recomputation", "s_recv": s_recv,
            "bins": list(bins), "ranks": ranks}


def layer_bound_ms(prof, peak_tflops):
    """Sum over the step's kernels of max(flops / MFMA peak, bytes / HBM peak):
    the step time at the roofline of every kernel."""
    return sum(max(v["flops"] / (peak_tflops * 1e12), v["bytes"] / (PEAK_HBM_GBS * 1e9)) * 1e3
               for v in prof.values())


def bench_router(mf, torch, w, dev, layer_step, steps, E_r):
    """Router forward and backward at the workload's shapes with E_r logits
    per token (HBM-bound: achieved algorithmic GB/s against 8 TB/s), and the
    trainable block router -> chunked layer -> layer backward -> router
    backward in tokens/s."""
    dt = dev["X"].dtype
    shape = mf.make_shape(w.T, w.h, w.F, E_r, w.k, mf.BF16 if w.dtype == "bf16" else mf.F32)
    gen = torch.Generator(device="cuda").manual_seed(4242)
    Wr = (torch.randn((E_r, w.h), generator=gen, device="cuda") / w.h ** 0.5).to(dt)
    idx = torch.empty((w.T, w.k), dtype=torch.int32, device="cuda")
    gates = torch.empty((w.T, w.k), device="cuda")
    dgr = torch.randn((w.T, w.k), generator=gen, device="cuda")
    dXr = torch.zeros((w.T, w.h), dtype=dt, device="cuda")
    dWr = torch.empty((E_r, w.h), device="cuda")

    def fwd_bwd():
        mf.memfine_router_fwd(shape, dev["X"], Wr, idx, gates)
        mf.memfine_router_bwd(shape, dev["X"], Wr, idx, gates, dgr, dXr, dWr,
                              accumulate_dX=True)

    for _ in range(3):
        fwd_bwd()
    torch.cuda.synchronize()
    names = ["router_fwd", "router_bwd_dx", "router_wgrad", "router_reduce"]
    mf.memfine_profile_begin(names)
    for _ in range(steps):
        fwd_bwd()
    torch.cuda.synchronize()
    prof = mf.memfine_profile_end()
    kern = {}
    for k in names:
        v = prof.get(k)
        if not v or not v["launches"]:
            continue
        ms = v["total_ms"] / v["launches"]
        gbs = v["bytes"] / v["launches"] / (ms * 1e-3) / 1e9
        kern[k] = {"avg_ms": round(ms, 4), "gbs": round(gbs, 1),
                   "hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
                   "tflops": round(v["flops"] / v["launches"] / (ms * 1e-3) / 1e12, 2)}
    # the block: router forward, layer, router backward into the layer's dX
    for _ in range(2):
        fwd_bwd()
        layer_step()
    torch.cuda.synchronize()
    a = time.perf_counter()
    for _ in range(steps):
        mf.memfine_router_fwd(shape, dev["X"], Wr, idx, gates)
        layer_step()
        mf.memfine_router_bwd(shape, dev["X"], Wr, idx, gates, dgr, dXr, dWr,
                              accumulate_dX=True)
    torch.cuda.synchronize()
    block_s = (time.perf_counter() - a) / steps
    log(f"[bench] router: " + ", ".join(f"{k} {v['avg_ms']:.4f} ms {v['gbs']:.0f} GB/s"
                                         for k, v in kern.items())
        + f"; block {w.T / block_s:.0f} tokens/s")
    return {"router_experts": E_r, "kernels": kern, "block_tokens_per_s": round(w.T / block_s, 1),
            "block_ms_per_step": round(block_s * 1e3, 4),
            "note": "router fwd + chunked layer fwd/bwd (same plan as the headline step) + "
                    "router bwd accumulating into dX; the layer's routing stays the "
                    "workload's seeded routing"}


def host_cpu():
    """CPU model and the BLAS library NumPy calls (for the oracle's timing)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        libs = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if libs:
            blas = f"{libs[0].get('internal_api')} {libs[0].get('version')}"
    except Exception:
        pass
    return {"model": model, "blas": blas}


def cpu_baseline(w, idx_np, gates_np, dev, C, target_s):
    """The oracle, as it stands, on the host: fp64 fwd + chunked-recompute bwd
    over the first T_s tokens (same weights, same chunk count)."""
    import torch

    from oracle import moe as om
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    log("[bench] cpu baseline: copying weights to host")
    W1 = dev["W1"].double().cpu().numpy()
    W2 = dev["W2"].double().cpu().numpy()
    Ts = max(16, min(w.T, 256))
    elapsed = 0.0
    while True:
        X = dev["X"][:Ts].double().cpu().numpy()
        dY = dev["dY"][:Ts].double().cpu().numpy()
        a = time.perf_counter()
        om.moe_fwd(X, idx_np[:Ts], gates_np[:Ts], W1, W2, C)
        om.moe_bwd(X, idx_np[:Ts], gates_np[:Ts], W1, W2, dY, C)
        elapsed = time.perf_counter() - a
        log(f"[bench] cpu baseline: {Ts} tokens in {elapsed:.2f} s")
        if elapsed >= target_s / 3 or Ts >= w.T:
            break
        Ts = min(w.T, int(Ts * max(2.0, target_s / max(elapsed, 1e-3))))
    out = {"value": round(Ts / elapsed, 2), "unit": "tokens/s", "cores": threads,
           "kind": "oracle", "cpu": host_cpu(),
           "sample": f"first {Ts} of {w.T} tokens, fp64 NumPy oracle fwd + chunked-recompute "
                     f"bwd at C={C}, {elapsed:.1f} s"}
    if w.h * w.F <= 2048 * 1408:
        # the small workloads also on one host thread, on a sample sized for
        # about a third of the time budget at the measured many-thread rate
        try:
            from threadpoolctl import threadpool_limits
            T1 = max(16, min(Ts, int(Ts / elapsed * target_s / 3 / max(threads, 1))))
            with threadpool_limits(limits=1):
                X = dev["X"][:T1].double().cpu().numpy()
                dY = dev["dY"][:T1].double().cpu().numpy()
                a = time.perf_counter()
                om.moe_fwd(X, idx_np[:T1], gates_np[:T1], W1, W2, C)
                om.moe_bwd(X, idx_np[:T1], gates_np[:T1], W1, W2, dY, C)
                e1 = time.perf_counter() - a
            out["one_thread"] = {"value": round(T1 / e1, 2), "unit": "tokens/s", "cores": 1,
                                 "sample": f"first {T1} of {w.T} tokens, {e1:.1f} s"}
            log(f"[bench] cpu baseline, one thread: {T1} tokens in {e1:.2f} s")
        except ImportError:
            pass
    del W1, W2
    torch.cuda.synchronize()
    return out


if __name__ == "__main__":
    main()
