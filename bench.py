#!/usr/bin/env python3
"""Benchmark: simulated replica-iterations per second on one MI355X.

The benchmark workload is the largest single-GPU configuration: Nested WAIT
on a heavy-tailed 10-type mix (prompt lengths the decile medians of
LogNormal(6, 0.8), output lengths clamp(ceil(LogNormal(5.5, 1.0)), 1, 4096),
segments (128, 256, 512, 1024, 2048, 4096), thresholds 1, KV budget 262144
tokens, iteration time 15 ms + 0.05 ms/token, rate 0.9x the fluid stability
boundary), 8192 replicas x 1e6 batches = 8.19e9 replica-iterations.

The job's horizon is split over the timed steps: step i advances every
replica by its share of the horizon, resuming from the state the previous
step left (step 0 starts from the empty system), so the K timed steps
together run the whole job once.  Warmup steps run the same chunks on a
separate workspace.  Job tables are copied to HBM before the timed region.

Prints one JSON line.  The roofline object prices the simulation kernel
against the ALU peak with an explicit operation model (lane-operations the
method needs per arrival, batch, completion, eviction and idle wait) and
against the HBM peak with the record-traffic model (32 bytes per arrival and
per completion), both from the event counts the kernel itself returns; the
larger fraction binds.  The cpu_baseline object times the CPU oracle on a
bounded sample of the same workload on the host threads the box allots.
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
    """Record traffic the method needs: 32 bytes per arrival and per
    completion (a request record written when it queues and read when it
    leaves, both ends of its life)."""
    return float(32 * (res["arrivals"].sum() + res["completions"].sum()))


def chunks(horizon: int, steps: int):
    """Split a horizon into `steps` consecutive chunks (sizes differ by at most
    one batch)."""
    return [(i + 1) * horizon // steps - i * horizon // steps for i in range(steps)]


def host_cpu() -> dict:
    """The host's CPU model, logical CPU count and the CPUs this process may
    run on."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        allowed = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        allowed = os.cpu_count() or 1
    return {"model": model, "nproc": os.cpu_count() or 1, "allowed": allowed}


def baseline_threads() -> int:
    """Oracle threads: the CPUs this process may use, capped by the per-GPU
    thread allotment the environment states (OMP_NUM_THREADS), else 16."""
    cap = 16
    try:
        cap = max(1, int(os.environ.get("OMP_NUM_THREADS", "16")))
    except ValueError:
        pass
    return max(1, min(host_cpu()["allowed"], cap))


def source_hash(workload: str = "wait-llama") -> str:
    """Hash of the kernel sources a profiled workload runs and of the hipcc
    options they are compiled with."""
    from paper_2504_11320_amd import build as Bd
    h = hashlib.sha256()
    for name in PROFILES[workload][1]:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
        if name.endswith(".hip"):
            h.update(" ".join(Bd.flags_for(name)).encode())
    return h.hexdigest()[:16]


def traffic_from_profile(workload: str, rep_its_per_launch: float):
    """Measured HBM bytes per launch: the DRAM bytes per replica-iteration of
    the workload's committed rocprofv3 counter summary, times the
    replica-iterations of one launch here; None if there is no summary or it
    was not taken on the current kernel sources."""
    if workload not in PROFILES:
        return None
    path = os.path.join(ROOT, "profiles", PROFILES[workload][0] + "_hbm.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    h = re.search(r"source_sha256_16:\s*([0-9a-f]+)", txt)
    b = re.search(r"hbm_bytes_per_replica_iteration:\s*([0-9.eE+]+)", txt)
    if not h or not b or h.group(1) != source_hash(workload):
        return None
    return float(b.group(1)) * rep_its_per_launch


# Workloads this script can time (the first is the benchmark's).  Each entry:
# (description, job builder, horizon, policy, jobs sampled by the CPU
# baseline, replicas of each sampled job the CPU baseline runs)
def _workloads():
    import workloads as W
    return {
        "nested-heavytail": ("Nested WAIT, heavy-tailed 10-type mix: prompts the decile "
                             "medians of LogNormal(6, 0.8), outputs clamp(ceil(LogNormal"
                             "(5.5, 1.0)), 1, 4096), segments (128, 256, 512, 1024, 2048, "
                             "4096), thresholds 1, C = 262144, 0.9x the fluid boundary, "
                             "8192 replicas x 1e6 batches",
                             lambda reps: W.config5(), 1000000, "nested", [0], 128),
        "wait-llama": ("WAIT, Llama-2-7B-shaped 3-type synthetic mix, 32 rates "
                       "0.5-1.2x fluid boundary, 1024 replicas each",
                       lambda reps: W.config2(replicas=reps), 100000, "wait", [0, 31], 256),
        "nested-geometric": ("Nested WAIT, 3 types, geometric outputs capped at 2048, "
                             "segments (64,256,1024,2048), 32 rates x 1024 replicas",
                             lambda reps: W.config3(replicas=reps), 100000, "nested", [0, 31],
                             128),
        "wait-sweep": ("WAIT threshold grid 16x16 x 16 rates x 16 replicas plus FCFS "
                       "on the same streams",
                       lambda reps: W.config4(), 100000, "wait+fcfs", [0, 4096], 16),
        "nowait-llama": ("WAIT-no-wait (thresholds 1, 1, 1) on the Llama-2-7B-shaped "
                         "3-type mix, 32 rates 0.5-1.2x fluid boundary, 1024 replicas each",
                         lambda reps: _nowait(W.config2(replicas=reps)), 100000,
                         "wait-nowait", [0, 31], 256),
        "wait-cyclic": ("WAIT on the Llama-2-7B-shaped 3-type mix with cyclic "
                        "time-varying rates lam_j (1 + 0.5 sin(4 pi t / 8e8 ms + 2 pi j / 3)), "
                        "32 rates 0.5-1.2x fluid boundary, 1024 replicas each",
                        lambda reps: W.config_cyclic(replicas=reps), 100000, "wait", [0, 31],
                        256),
        "pd-decode": ("decode-only p630d20 (PD-disaggregated decode server: 630-token "
                      "context, 20 generated tokens), WAIT with fluid thresholds and FCFS "
                      "with a 1% reserve, 9 rates 0.1-0.5/ms, 1024 replicas each",
                      lambda reps: W.config_pd(replicas=reps), 100000, "wait+fcfs", [8, 17],
                      64),
        "fcfs-chunked": ("FCFS with a 1% reserve and 512-token chunked prefill (the "
                         "Sarathi-style baseline) on the Llama-2-7B-shaped 3-type mix, 32 "
                         "rates 0.5-1.2x fluid boundary, 1024 replicas each",
                         lambda reps: W.config_chunked(replicas=reps), 100000, "fcfs",
                         [0, 31], 256),
        "wait-small": ("WAIT, 2 types (16/8, 32/16), C = 2048, 64 replicas",
                       lambda reps: W.config1(), 10000, "wait", [0], 64),
    }


def _nowait(jobs):
    for j in jobs:
        j.wl.policy = "wait-nowait"
    return jobs


def cpu_baseline(jobs, pick, horizon: int, replicas: int, threads: int) -> dict:
    """The oracle on a bounded sample: `replicas` replicas of each picked job
    over the first min(horizon, 1e5) batches."""
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
    cpu = host_cpu()
    return {"value": total / dt, "unit": UNIT, "cores": threads, "kind": "oracle",
            "sample": f"jobs {pick} of {len(jobs)} x {n} replicas x {horizon} batches "
                      f"({total} replica-iterations, {dt:.1f} s)",
            "cpu_model": cpu["model"], "nproc": cpu["nproc"], "cpus_allowed": cpu["allowed"]}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="nested-heavytail",
                    help="nested-heavytail (the benchmark), wait-llama, nested-geometric, "
                         "wait-sweep, nowait-llama, wait-cyclic, pd-decode, fcfs-chunked, "
                         "wait-small")
    ap.add_argument("--horizon", type=int, default=0,
                    help="batches per replica over all timed steps (0: the workload's)")
    ap.add_argument("--replicas", type=int, default=1024)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-replicas", type=int, default=0,
                    help="replicas per sampled job in the CPU baseline (0: the workload's)")
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
    if args.steps < 1:
        print("bench.py: --steps must be at least 1", file=sys.stderr)
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
    desc, build, horizon0, policy, pick, cpu_reps = table[args.workload]
    horizon = args.horizon or horizon0
    jobs = build(args.replicas)
    m = max(j.wl.m for j in jobs)
    cdf_cap = max((j.wl.out_cap for j in jobs if j.wl.out_cdf is not None), default=0)
    rate_pts = max((len(j.wl.rate_t) for j in jobs if j.wl.rate_t is not None), default=0)
    cpa = candidates_per_arrival(jobs)
    parts = chunks(horizon, args.steps)
    stream = torch.cuda.current_stream()

    if args.warmup > 0:  # the same chunks on a workspace of its own
        warm = B.Simulation(jobs)
        warm.prepare()
        for i in range(args.warmup):
            warm.advance(parts[i % len(parts)], resume=i > 0)
        torch.cuda.synchronize()
        del warm
        torch.cuda.empty_cache()

    sim = B.Simulation(jobs)
    sim.prepare()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    t0 = time.perf_counter()
    for i, h in enumerate(parts):
        sim.advance(h, resume=i > 0)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = ev0.elapsed_time(ev1)
    ms_step = ms_total / args.steps

    res = sim.results()
    rep_its = int(res["batches"].sum())
    if rep_its != len(res["batches"]) * horizon or np.any(res["flags"] & 3):
        print("bench.py: some replicas stopped early (flags set)", file=sys.stderr)
    value = rep_its / (ms_total / 1e3)

    # Roofline of the simulation kernel: algorithmic work of the whole job
    # over the time of its launches (one launch per step).
    secs = ms_total / 1e3
    ops = algorithmic_ops(res, m, cdf_cap, rate_pts, cpa)
    nbytes = algorithmic_bytes(res)
    alu = {"achieved": ops / secs, "peak": ALU_PEAK, "unit": "lane-ops/s"}
    hbm = {"achieved": nbytes / secs, "peak": HBM_PEAK, "unit": "B/s"}
    alu["frac"] = alu["achieved"] / ALU_PEAK
    hbm["frac"] = hbm["achieved"] / HBM_PEAK
    bind, bound = (alu, "alu") if alu["frac"] >= hbm["frac"] else (hbm, "hbm")
    full = args.horizon in (0, horizon0) and args.replicas == 1024
    traffic = traffic_from_profile(args.workload, rep_its / args.steps) if full else None
    roofline = {"bound": bound, "achieved": bind["achieved"], "peak": bind["peak"],
                "unit": bind["unit"], "frac": bind["frac"],
                # measured DRAM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE,
                # scaled by a plain copy's counters), null if not taken on these sources
                "traffic": traffic,
                "alu_frac": alu["frac"], "hbm_frac": hbm["frac"],
                "algorithmic_ops_per_replica_iteration": ops / rep_its,
                "algorithmic_bytes_per_replica_iteration": nbytes / rep_its,
                "hbm_measured_frac": (traffic * args.steps / secs / HBM_PEAK
                                      if traffic is not None else None),
                "launches": args.steps,
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
                      "horizon_batches": horizon, "batches_per_step": parts[0],
                      "replica_iterations": rep_its, "policy": policy,
                      "kv_budget_tokens": int(max(j.wl.C for j in jobs))},
           "roofline": roofline,
           "wall_s_timed": wall}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(jobs, pick, horizon, args.cpu_replicas or cpu_reps,
                                           baseline_threads())
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
