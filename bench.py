#!/usr/bin/env python3
"""Benchmark: simulated replica-iterations per second on one MI355X.

One step is one pass of the whole simulation over the benchmark workload:
the Llama-2-7B-shaped WAIT workload (3 request types, prompts 128/512/1024,
outputs 64/256/512, mix 0.5/0.3/0.2, KV budget 131072 tokens, iteration time
15 ms + 0.05 ms/token, thresholds (1,1,1)) at 32 arrival rates spanning
0.5-1.2x the fluid stability boundary, 1024 replicas per rate, 1e5 batches
per replica: 3.2768e9 replica-iterations per step.  Inputs (job tables) are
copied to HBM before the timed region; every replica starts from the empty
system in every step.

Prints one JSON line.  The roofline object prices the simulation kernel
against the ALU peak with an explicit operation model (lane-operations the
method needs per arrival, batch, completion, eviction and idle wait; see the
design notes), using the event counts the kernel itself returns.  The
cpu_baseline object times the CPU oracle on a bounded sample of the same
workload (2 rates x 256 replicas x the full horizon) on the host's cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "simulated replica-iterations/sec (1 GPU) + % of VALU/HBM roofline"
UNIT = "replica-iterations/s"

# MI355X: 256 compute units x 4 SIMD x 16 lanes per clock at 2.4 GHz = 64
# lane-operations per CU per clock (full-rate VALU, fp64 included).
CUS, LANES_PER_CU_CLK, CLOCK_HZ = 256, 64, 2.4e9
ALU_PEAK = CUS * LANES_PER_CU_CLK * CLOCK_HZ          # 3.93e13 lane-ops/s
HBM_PEAK = 8.0e12                                     # bytes/s

CSRC = os.path.join(ROOT, "paper_2504_11320_amd", "csrc")
# Per workload: the committed rocprofv3 HBM counter summary of its dominant
# kernel and the sources that define that kernel (hashed to tie the summary
# to the kernel it was measured on).
_WAIT_SRCS = ("sim_known_impl.h", "sim_known_wait.hip", "sim_common.h")
PROFILES = {
    "wait-llama": ("sim_known_wait_3type_32x1024x1e5", _WAIT_SRCS),
    "wait-cyclic": ("sim_known_wait_tv_3type_cyclic_32x1024x1e5",
                    ("sim_known_impl.h", "sim_known_wait_tv.hip", "sim_common.h")),
    "nested-geometric": ("sim_nested_3type_geometric_32x1024x1e5",
                         ("sim_nested_impl.h", "sim_nested.hip", "sim_common.h")),
    "nested-heavytail": ("sim_nested_10type_lognormal_8192x1e6",
                         ("sim_nested_impl.h", "sim_nested.hip", "sim_common.h")),
    "fcfs-chunked": ("sim_known_fcfs_3type_chunk512_32x1024x1e5",
                     ("sim_known_impl.h", "sim_known_fcfs.hip", "sim_common.h")),
}


def op_model(m: int, cdf_cap: int = 0, rate_pts: int = 0, cand_per_arrival: float = 1.0) -> dict:
    """Algorithmic lane-operations per event (full-rate VALU instruction
    equivalents; a 32x32->64-bit multiply counts 4).  cdf_cap > 1: output
    lengths are drawn from a CDF table of that many entries (a search of
    2 ops per halving step).  rate_pts > 0: time-varying rates sampled by
    thinning, cand_per_arrival candidates drawn per arrival, each tested
    against the profile (a search over its points, one interpolation)."""
    philox = 10 * (2 * 4 + 4 + 2)     # 2 wide multiplies, 4 xor, 2 key adds per round
    uniform = 10                      # 52-bit assembly, int->fp64, scale
    ln = 50                           # reduction, one fp64 division, 12-term Horner, e*ln2
    gap = 14                          # fp64 division by lambda, add to the clock
    book = 12                         # queue push, counters, area terms
    cdf = 2 * max(0, int(cdf_cap - 1).bit_length()) if cdf_cap > 1 else 0
    cand = philox + uniform + ln + gap + cdf
    if rate_pts > 0:
        # search (compare, select per halving step), fp64 division and
        # interpolation, w3 * fmax and the comparison, zero-stretch tests
        cand += 3 * max(1, int(rate_pts - 1).bit_length()) + 14 + 4 + 6
    return {
        "arrival": cand_per_arrival * cand + book + 2 * m,
        "batch": 24 + 6 * m,          # eligibility, tokens, tau, clock, areas, peak
        "completion": 35,             # latency, sum, histogram search and update
        "eviction": 14 + 3 * m,       # LIFO choice, stage, memory, re-queue
        "idle": 15 + 4 * m,           # next arrival, area terms, eligibility
    }


def candidates_per_arrival(jobs) -> float:
    """Thinning draws lam_j max f_j candidates per unit time for lam_j f_j
    arrivals: the ratio of the bound to the profile's mean over its span,
    weighted by the rates (1 for constant rates)."""
    import numpy as np
    bound = mean = 0.0
    for j in jobs:
        wl = j.wl
        for k in range(wl.m):
            if wl.rate_t is None or len(wl.rate_t) < 2:
                bound += wl.lam[k] * j.n
                mean += wl.lam[k] * j.n
                continue
            f = np.asarray(wl.rate_f, dtype=np.float64).reshape(wl.m, -1)[k]
            t = np.asarray(wl.rate_t, dtype=np.float64)
            fbar = float(np.sum(np.diff(t) * (f[1:] + f[:-1]) / 2.0) / (t[-1] - t[0]))
            bound += wl.lam[k] * f.max() * j.n
            mean += wl.lam[k] * fbar * j.n
    return bound / mean if mean > 0 else 1.0


def algorithmic_ops(res: dict, m: int, cdf_cap: int = 0, rate_pts: int = 0,
                    cand_per_arrival: float = 1.0) -> float:
    c = op_model(m, cdf_cap, rate_pts, cand_per_arrival)
    return float(c["batch"] * res["batches"].sum() + c["arrival"] * res["arrivals"].sum()
                 + c["completion"] * res["completions"].sum()
                 + c["eviction"] * res["evictions"].sum() + c["idle"] * res["idle_waits"].sum())


def algorithmic_bytes(res: dict) -> float:
    """Record traffic the method needs: 16 B written and read per queued
    request (arrival and re-queue) and per admission/completion."""
    ev = res["arrivals"].sum() + res["evictions"].sum()
    return float(16 * 2 * ev + 16 * res["completions"].sum())


def source_hash(workload: str = "wait-llama") -> str:
    h = hashlib.sha256()
    for name in PROFILES[workload][1]:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_from_profile(workload: str):
    """HBM bytes per launch from the workload's committed rocprofv3 counter
    summary, if there is one and it was taken on the current kernel source."""
    if workload not in PROFILES:
        return None
    path = os.path.join(ROOT, "profiles", PROFILES[workload][0] + "_hbm.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    h = re.search(r"source_sha256_16:\s*([0-9a-f]+)", txt)
    b = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    if not h or not b or h.group(1) != source_hash(workload):
        return None
    return float(b.group(1))


# Workloads this script can time (the first is the benchmark's).  Each entry:
# (description, job builder, horizon, policy, jobs sampled by the CPU baseline)
def _workloads():
    import workloads as W
    return {
        "wait-llama": ("WAIT, Llama-2-7B-shaped 3-type synthetic mix, 32 rates "
                       "0.5-1.2x fluid boundary, 1024 replicas each",
                       lambda reps: W.config2(replicas=reps), 100000, "wait", [0, 31]),
        "nested-geometric": ("Nested WAIT, 3 types, geometric outputs capped at 2048, "
                             "segments (64,256,1024,2048), 32 rates x 1024 replicas",
                             lambda reps: W.config3(replicas=reps), 100000, "nested", [0, 31]),
        "wait-sweep": ("WAIT threshold grid 16x16 x 16 rates x 16 replicas plus FCFS "
                       "on the same streams",
                       lambda reps: W.config4(), 100000, "wait+fcfs", [0, 4096]),
        "nested-heavytail": ("Nested WAIT, 10 lognormal-decile prompt types, lognormal "
                             "outputs capped at 4096, 6 segments, 8192 replicas",
                             lambda reps: W.config5(), 1000000, "nested", [0]),
        "nowait-llama": ("WAIT-no-wait (thresholds 1, 1, 1) on the Llama-2-7B-shaped "
                         "3-type mix, 32 rates 0.5-1.2x fluid boundary, 1024 replicas each",
                         lambda reps: _nowait(W.config2(replicas=reps)), 100000,
                         "wait-nowait", [0, 31]),
        "wait-cyclic": ("WAIT on the Llama-2-7B-shaped 3-type mix with cyclic "
                        "time-varying rates lam_j (1 + 0.5 sin(4 pi t / 8e8 ms + 2 pi j / 3)), "
                        "32 rates 0.5-1.2x fluid boundary, 1024 replicas each",
                        lambda reps: W.config_cyclic(replicas=reps), 100000, "wait", [0, 31]),
        "pd-decode": ("decode-only p630d20 (PD-disaggregated decode server: 630-token "
                      "context, 20 generated tokens), WAIT with fluid thresholds and FCFS "
                      "with a 1% reserve, 9 rates 0.1-0.5/ms, 1024 replicas each",
                      lambda reps: W.config_pd(replicas=reps), 100000, "wait+fcfs", [8, 17]),
        "fcfs-chunked": ("FCFS with a 1% reserve and 512-token chunked prefill (the "
                         "Sarathi-style baseline) on the Llama-2-7B-shaped 3-type mix, 32 "
                         "rates 0.5-1.2x fluid boundary, 1024 replicas each",
                         lambda reps: W.config_chunked(replicas=reps), 100000, "fcfs",
                         [0, 31]),
        "wait-small": ("WAIT, 2 types (16/8, 32/16), C = 2048, 64 replicas",
                       lambda reps: W.config1(), 10000, "wait", [0]),
    }


def _nowait(jobs):
    for j in jobs:
        j.wl.policy = "wait-nowait"
    return jobs


def cpu_baseline(jobs, pick, horizon: int, replicas: int, threads: int) -> dict:
    """The oracle on a bounded sample: `replicas` replicas of each picked job,
    the full horizon (at most 1e5 batches)."""
    from oracle import oracle as O
    import numpy as np
    import workloads as W
    horizon = min(horizon, 100000)
    t0 = time.perf_counter()
    total = 0
    for i in pick:
        job = jobs[i]
        sub = W.Job(job.wl, job.seed, np.asarray(job.replica_ids[:replicas], dtype=np.uint32))
        r = O.run_job(sub, horizon, threads=threads)
        total += int(r["batches"].sum())
    dt = time.perf_counter() - t0
    n = min(replicas, min(jobs[i].n for i in pick))
    return {"value": total / dt, "unit": UNIT, "cores": threads, "kind": "oracle",
            "sample": f"jobs {pick} of {len(jobs)} x {n} replicas x {horizon} batches "
                      f"({total} replica-iterations, {dt:.1f} s)"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="wait-llama",
                    help="wait-llama (the benchmark), nested-geometric, wait-sweep, "
                         "nested-heavytail, nowait-llama, wait-cyclic, pd-decode, "
                         "fcfs-chunked, wait-small")
    ap.add_argument("--horizon", type=int, default=0, help="batches (0: the workload's)")
    ap.add_argument("--replicas", type=int, default=1024)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-replicas", type=int, default=256)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (used to "
                         "scale the HBM byte counters)")
    args = ap.parse_args()

    if args.copy_calibration:
        import torch
        n = args.copy_calibration << 20
        a = torch.ones(n, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "launches": 3}))
        return 0

    if args.gpus != 1:
        print(f"bench.py: this simulator runs on one GPU; --gpus {args.gpus} is not "
              f"supported (replicas shard across GPUs with no communication; this "
              f"benchmark measures a single MI355X)", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    import workloads as W
    from paper_2504_11320_amd import binding as B

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    B.lib()  # fails loudly if the HIP library is missing

    table = _workloads()
    if args.workload not in table:
        print(f"bench.py: unknown workload {args.workload}", file=sys.stderr)
        return 2
    desc, build, horizon0, policy, pick = table[args.workload]
    args.horizon = args.horizon or horizon0
    jobs = build(args.replicas)
    m = max(j.wl.m for j in jobs)
    cdf_cap = max((j.wl.out_cap for j in jobs if j.wl.out_cdf is not None), default=0)
    rate_pts = max((len(j.wl.rate_t) for j in jobs if j.wl.rate_t is not None), default=0)
    cpa = candidates_per_arrival(jobs)
    sim = B.Simulation(jobs)
    sim.prepare()
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        sim.advance(args.horizon, resume=False)
    torch.cuda.synchronize()

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        sim.advance(args.horizon, resume=False)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = ev0.elapsed_time(ev1)
    ms_step = ms_total / args.steps

    res = sim.results()
    rep_its = int(res["batches"].sum())
    if rep_its != len(res["batches"]) * args.horizon or np.any(res["flags"] & 3):
        print("bench.py: some replicas stopped early (flags set)", file=sys.stderr)
    value = rep_its / (ms_step / 1e3)

    ops = algorithmic_ops(res, m, cdf_cap, rate_pts, cpa)
    achieved = ops / (ms_step / 1e3)
    full = args.horizon == horizon0 and args.replicas == 1024
    traffic = traffic_from_profile(args.workload) if full else None
    roofline = {"bound": "alu", "achieved": achieved, "peak": ALU_PEAK,
                "unit": "lane-ops/s", "frac": achieved / ALU_PEAK,
                "traffic": traffic,
                "algorithmic_ops_per_replica_iteration": ops / rep_its,
                "algorithmic_bytes_per_launch": algorithmic_bytes(res),
                # the HBM side of the same launch: algorithmic record bytes and
                # the measured DRAM bytes (traffic), each per second over the
                # 8 TB/s peak
                "hbm_algorithmic_frac": algorithmic_bytes(res) / (ms_step / 1e3) / HBM_PEAK,
                "hbm_measured_frac": (traffic / (ms_step / 1e3) / HBM_PEAK
                                      if traffic is not None else None),
                "kernel": (f"sim_nested_kernel ({m} types)" if policy == "nested"
                           else f"sim_known_kernel ({policy}, {m} types)")
                          + (f", time-varying rates ({rate_pts} points, "
                             f"{cpa:.3f} candidates per arrival)" if rate_pts else "")}

    out = {"metric": METRIC, "value": value, "unit": UNIT, "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "f64", "data": "synthetic",
           "config": {"workload": desc, "name": args.workload,
                      "replicas": len(res["batches"]), "jobs": len(jobs),
                      "horizon_batches": args.horizon,
                      "replica_iterations_per_step": rep_its, "policy": policy,
                      "kv_budget_tokens": int(max(j.wl.C for j in jobs))},
           "roofline": roofline,
           "wall_s_timed": wall}
    if not args.no_cpu_baseline:
        threads = max(1, min(os.cpu_count() or 1, 16))
        out["cpu_baseline"] = cpu_baseline(jobs, pick, args.horizon, args.cpu_replicas, threads)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
