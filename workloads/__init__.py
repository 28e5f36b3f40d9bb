"""Seeded synthetic workloads for the simulator and its oracle.

This module only describes inputs: request types, Poisson rates, iteration
time constants, KV budgets, thresholds, segment boundaries, output-length CDF
tables, latency histogram edges and replica streams.  It holds none of the
simulation's arithmetic, so both the GPU library's tests and the oracle can
draw their inputs from it.

Rates are given per millisecond, times in milliseconds, lengths in tokens.
Each sweep is expressed relative to a rate scale LAM_STAR_*: the total arrival
rate at which the fluid memory requirement of the mix equals the KV budget
(Section 3.2 of arXiv 2504.11320).  The literals below were computed once from
that definition; a CPU test recomputes them with the fluid calculator.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

# ---------------------------------------------------------------- types ----


@dataclasses.dataclass
class Workload:
    """One simulated system: types, rates, time model, memory, policy."""

    prompt_len: List[int]
    lam: List[float]                 # Poisson rate per type, per ms
    d0: float                        # ms per iteration
    d1: float                        # ms per cached token
    C: int                           # KV budget, tokens
    policy: str                      # "wait" | "wait-nowait" | "nested" | "fcfs"
    n: List[int]                     # thresholds (WAIT: per type, Nested: per segment)
    out_len: Optional[List[int]] = None     # known output lengths, or None
    out_cap: int = 0                         # distribution mode: cap
    out_cdf: Optional[np.ndarray] = None     # uint32 [m, out_cap-1]
    seg_end: Optional[List[int]] = None      # Nested: r_1 < ... < r_L
    reserve: float = 0.0                     # FCFS admission reserve (fraction of C)
    chunk: int = 0                           # FCFS prefill tokens per iteration (0: whole)
    hist_edges: Optional[np.ndarray] = None  # latency histogram edges (ms)
    record_capacity: int = 1 << 15           # external-queue capacity
    trace: Optional[tuple] = None            # (times f64, types i32, lengths i32)
    # time-varying rates: type j arrives at lam[j] * f_j(t), f_j piecewise
    # linear through (rate_t[i], rate_f[j][i]) and constant outside
    rate_t: Optional[np.ndarray] = None      # f64 [P], strictly increasing
    rate_f: Optional[np.ndarray] = None      # f64 [m, P], >= 0
    # Nested WAIT per-stage caps: cap of decode stage s at index s - 1
    # (seg_end[-1] entries); segment k's caps are taken in turn, one per
    # service, as the size of its entering cohort; n[k] is the largest
    stage_caps: Optional[List[int]] = None

    @property
    def m(self) -> int:
        return len(self.prompt_len)


@dataclasses.dataclass
class Job:
    """A workload run on a set of replica streams."""

    wl: Workload
    seed: int
    replica_ids: np.ndarray          # uint32

    @property
    def n(self) -> int:
        return int(len(self.replica_ids))


def default_edges(d0: float, count: int = 192) -> np.ndarray:
    """Latency histogram edges d0 * 2^(b/8), b = 0..count-1."""
    return np.array([d0 * 2.0 ** (b / 8.0) for b in range(count)], dtype=np.float64)


def ids(n: int, start: int = 0) -> np.ndarray:
    return np.arange(start, start + n, dtype=np.uint32)


# -------------------------------------------------- output distributions ----


def _cdf_table(F: Sequence[float]) -> np.ndarray:
    """u32 thresholds T[s] = min(2^32-1, floor(2^32 F(s))), s = 1..cap-1."""
    out = np.empty(len(F), dtype=np.uint32)
    for i, f in enumerate(F):
        out[i] = min(0xFFFFFFFF, int(math.floor(f * 4294967296.0)))
    return out


def geometric_cdf_table(mean: float, cap: int) -> np.ndarray:
    """P(L=k) = (1/mean)(1-1/mean)^(k-1) for k < cap, tail mass at cap."""
    q = 1.0 - 1.0 / mean
    return _cdf_table([1.0 - q ** s for s in range(1, cap)])


def lognormal_cdf_table(mu: float, sigma: float, cap: int) -> np.ndarray:
    """L = clamp(ceil(X), 1, cap), X ~ LogNormal(mu, sigma)."""
    F = [0.5 * (1.0 + math.erf((math.log(s) - mu) / (sigma * math.sqrt(2.0))))
         for s in range(1, cap)]
    return _cdf_table(F)


def lognormal_decile_medians(mu: float, sigma: float) -> List[int]:
    """Prompt lengths: medians of the ten deciles of LogNormal(mu, sigma)."""
    from statistics import NormalDist
    nd = NormalDist()
    return [int(round(math.exp(mu + sigma * nd.inv_cdf((i + 0.5) / 10.0))))
            for i in range(10)]


# ------------------------------------------------------------ configs ----

# Total rate (per ms) at which the fluid memory of each mix equals C.
LAM_STAR_C2 = 0.00010735521308933886   # 3-type Llama-shaped mix, C = 131072
LAM_STAR_C3 = 9.235201143089613e-05    # same prompts, geometric outputs
LAM_STAR_C5 = 4.891271666677714e-05    # 10-type heavy-tailed mix, C = 262144

C2_PROMPTS = [128, 512, 1024]
C2_OUTPUTS = [64, 256, 512]
C2_MIX = [0.5, 0.3, 0.2]


def config1(replicas: int = 64, record_capacity: int = 1 << 17) -> List[Job]:
    """WAIT, known lengths, 2 types (16/8, 32/16), lam = (0.4, 0.2)/ms,
    5 ms + 0.01 ms/token, C = 2048, thresholds (4, 2)."""
    wl = Workload(prompt_len=[16, 32], lam=[0.4, 0.2], d0=5.0, d1=0.01, C=2048,
                  policy="wait", n=[4, 2], out_len=[8, 16],
                  hist_edges=default_edges(5.0), record_capacity=record_capacity)
    return [Job(wl, 0, ids(replicas))]


def c2_rates(n_rates: int = 32) -> List[float]:
    return [LAM_STAR_C2 * (0.5 + 0.7 * i / (n_rates - 1)) for i in range(n_rates)]


def config2(replicas: int = 1024, n_rates: int = 32, rate_index=None,
            record_capacity: int = 1 << 15) -> List[Job]:
    """WAIT, Llama-2-7B-shaped synthetic: 3 types, prompts (128, 512, 1024),
    outputs (64, 256, 512), mix (0.5, 0.3, 0.2), C = 131072,
    15 ms + 0.05 ms/token, thresholds (1, 1, 1), rates spanning 0.5-1.2x the
    fluid boundary."""
    jobs = []
    rates = c2_rates(n_rates)
    sel = range(n_rates) if rate_index is None else rate_index
    for i in sel:
        lam = [p * rates[i] for p in C2_MIX]
        wl = Workload(prompt_len=list(C2_PROMPTS), lam=lam, d0=15.0, d1=0.05,
                      C=131072, policy="wait", n=[1, 1, 1],
                      out_len=list(C2_OUTPUTS), hist_edges=default_edges(15.0),
                      record_capacity=record_capacity)
        jobs.append(Job(wl, 0, ids(replicas)))
    return jobs


def config3(replicas: int = 1024, n_rates: int = 32, rate_index=None,
            record_capacity: int = 1 << 15) -> List[Job]:
    """Nested WAIT, unknown outputs: C2's prompts and mix, outputs geometric
    with means (64, 256, 512) capped at 2048, segments (64, 256, 1024, 2048),
    thresholds 1 per segment, C = 131072."""
    cap = 2048
    cdf = np.stack([geometric_cdf_table(mu, cap) for mu in (64, 256, 512)])
    jobs = []
    sel = range(n_rates) if rate_index is None else rate_index
    for i in sel:
        rate = LAM_STAR_C3 * (0.5 + 0.7 * i / (n_rates - 1))
        lam = [p * rate for p in C2_MIX]
        wl = Workload(prompt_len=list(C2_PROMPTS), lam=lam, d0=15.0, d1=0.05,
                      C=131072, policy="nested", n=[1, 1, 1, 1], out_cap=cap,
                      out_cdf=cdf, seg_end=[64, 256, 1024, 2048],
                      hist_edges=default_edges(15.0),
                      record_capacity=record_capacity)
        jobs.append(Job(wl, 0, ids(replicas)))
    return jobs


def config4(replicas: int = 16, grid: int = 16, n_rates: int = 16,
            record_capacity: int = 1 << 14) -> List[Job]:
    """Policy sweep: WAIT thresholds (n1, n2) in {1..grid}^2, n3 = 1, at
    n_rates rates, plus FCFS (reserve 0) at the same rates, all on the same
    replica streams."""
    jobs = []
    for i in range(n_rates):
        rate = LAM_STAR_C2 * (0.5 + 0.7 * i / (n_rates - 1))
        lam = [p * rate for p in C2_MIX]
        for n1 in range(1, grid + 1):
            for n2 in range(1, grid + 1):
                wl = Workload(prompt_len=list(C2_PROMPTS), lam=lam, d0=15.0,
                              d1=0.05, C=131072, policy="wait", n=[n1, n2, 1],
                              out_len=list(C2_OUTPUTS),
                              hist_edges=default_edges(15.0),
                              record_capacity=record_capacity)
                jobs.append(Job(wl, 0, ids(replicas)))
    for i in range(n_rates):
        rate = LAM_STAR_C2 * (0.5 + 0.7 * i / (n_rates - 1))
        lam = [p * rate for p in C2_MIX]
        wl = Workload(prompt_len=list(C2_PROMPTS), lam=lam, d0=15.0, d1=0.05,
                      C=131072, policy="fcfs", n=[], out_len=list(C2_OUTPUTS),
                      hist_edges=default_edges(15.0),
                      record_capacity=record_capacity)
        jobs.append(Job(wl, 0, ids(replicas)))
    return jobs


def config5(replicas: int = 8192, record_capacity: int = 1 << 18) -> List[Job]:
    """Heavy-tailed 10-type mix: prompts = decile medians of LogNormal(6, 0.8),
    outputs clamp(ceil(LogNormal(5.5, 1.0)), 1, 4096), Nested WAIT with
    segments (128, 256, 512, 1024, 2048, 4096), thresholds 1, C = 262144,
    rate 0.9x the fluid boundary."""
    cap = 4096
    prompts = lognormal_decile_medians(6.0, 0.8)
    row = lognormal_cdf_table(5.5, 1.0, cap)
    cdf = np.stack([row] * len(prompts))
    rate = 0.9 * LAM_STAR_C5
    lam = [rate / len(prompts)] * len(prompts)
    wl = Workload(prompt_len=prompts, lam=lam, d0=15.0, d1=0.05, C=262144,
                  policy="nested", n=[1] * 6, out_cap=cap, out_cdf=cdf,
                  seg_end=[128, 256, 512, 1024, 2048, 4096],
                  hist_edges=default_edges(15.0), record_capacity=record_capacity)
    return [Job(wl, 0, ids(replicas))]


def config_chunked(replicas: int = 1024, n_rates: int = 32, chunk: int = 512,
                   record_capacity: int = 1 << 15) -> List[Job]:
    """The Sarathi-style baseline of Section 6 on the Llama-shaped mix:
    config2's types and rates under FCFS with a 1 % admission reserve and
    chunked prefill (at most `chunk` prefill tokens per iteration)."""
    jobs = []
    for j in config2(replicas, n_rates, None, record_capacity):
        wl = dataclasses.replace(j.wl, policy="fcfs", n=[], reserve=0.01, chunk=chunk)
        jobs.append(Job(wl, j.seed, j.replica_ids))
    return jobs


# ------------------------------------------- single-type p512d20 sweep ----

# The paper's single-type synthetic workload p512d20 (prompt 512, 20 decode
# tokens) in the linear time model: d0 = 10 ms and d1 chosen once so that the
# fluid boundary (the rate at which M* = C = 137,000 tokens) is 22 requests/s,
# the operating point the paper reports for WAIT on this workload.  Rates are
# fractions of that boundary; WAIT thresholds are ceil(n*) of the single-type
# fluid model at each rate (a CPU test recomputes them).
P512_LAMSTAR = 0.022                      # per ms
P512_D1 = 0.004073563169963875            # ms per cached token
P512_FRACS = [0.6, 0.7, 0.8, 0.85, 0.9, 0.95, 1.0]
P512_THRESHOLDS = [1, 1, 1, 2, 2, 4, 13]


def config_p512d20(replicas: int = 2048, record_capacity: int = 1 << 16) -> List[Job]:
    """p512d20 at 7 rates (0.6-1.0 of the fluid boundary) under WAIT (fluid
    thresholds), FCFS with a 1 % reserve, and FCFS with 512-token chunked
    prefill, on the same replica streams; job order: policy-major."""
    jobs = []
    for pol, chunk in (("wait", 0), ("fcfs", 0), ("fcfs", 512)):
        for frac, n in zip(P512_FRACS, P512_THRESHOLDS):
            wl = Workload(prompt_len=[512], lam=[frac * P512_LAMSTAR], d0=10.0, d1=P512_D1,
                          C=137000, policy=pol, n=[n] if pol == "wait" else [], out_len=[20],
                          reserve=0.01 if pol == "fcfs" else 0.0, chunk=chunk,
                          hist_edges=default_edges(10.0), record_capacity=record_capacity)
            jobs.append(Job(wl, 0, ids(replicas)))
    return jobs


# ------------------------------- two-type p512 mix under per-stage caps ----

# The paper's two-type workload (0.7 p512d20, 0.3 p512d50; prompt 512, outputs
# 20 or 50) under Nested WAIT with segments 1-20 and 21-50 and the per-stage
# caps that the batch-size cap tl = 30 gives (Section 6): continuation ratio
# 0.3, n_1 = 30 / (20 + 30 * 0.3), segment caps round(20 n_1) = 21 and
# round(9.31) = 9, spread as evenly as possible over the segments' 20 and 30
# decode stages (the first stages take one more).  A CPU test recomputes
# these caps from tl.  Time model and budget as p512d20.
P512MIX_SEG_END = [20, 50]
P512MIX_CAPS_TL30 = [2] + [1] * 19 + [1] * 9 + [0] * 21
P512MIX_RATES = [0.014, 0.018, 0.022]     # per ms


def config_p512_mix(replicas: int = 1024, rates=None, stage_caps=None,
                    record_capacity: int = 1 << 14) -> List[Job]:
    """The two-type p512 mix (outputs 20 or 50, unknown to the scheduler)
    under Nested WAIT with per-stage caps (default: those of tl = 30), one job
    per rate."""
    caps = list(P512MIX_CAPS_TL30 if stage_caps is None else stage_caps)
    cdf = _cdf_table([0.0] * 19 + [0.7] * 30)[None, :]
    n = [max(caps[:P512MIX_SEG_END[0]]), max(caps[P512MIX_SEG_END[0]:])]
    jobs = []
    for lam in (P512MIX_RATES if rates is None else rates):
        wl = Workload(prompt_len=[512], lam=[lam], d0=10.0, d1=P512_D1, C=137000,
                      policy="nested", n=n, out_cap=50, out_cdf=cdf,
                      seg_end=list(P512MIX_SEG_END), hist_edges=default_edges(10.0),
                      record_capacity=record_capacity, stage_caps=caps)
        jobs.append(Job(wl, 0, ids(replicas)))
    return jobs


# ------------------------------------- decode-only (PD-disaggregated) ----

# A decode server behind a separate prefill service receives each request with
# its context already cached (630 tokens) and generates 20 tokens.  In the
# model that is prompt length 630 and output length 19: the model's first
# processing (time and memory charge l) is the first decode step over the
# 630-token context, its stage s the step over 630 + s tokens, 20 processings
# per request; end-to-end latency is unchanged, a request's generated tokens
# are its model output length + 1, and its first token is the end of the first
# processing.  Time model 10 ms + 5e-5 ms per cached token, KV budget 137,000
# tokens (an A100 80 GB serving Llama-2-7B after weights and a 1 % margin).
PD_CONTEXT, PD_DECODE = 630, 20
PD_RATES = [0.10 + 0.05 * i for i in range(9)]     # 100-500 requests/s, per ms
# WAIT thresholds ceil(n*) with n* = lam d0 / (1 - d1 lam (l'+1)(l + l'/2))
# (single-type fluid model), computed once per rate; a CPU test recomputes them.
PD_THRESHOLDS = [2, 2, 3, 3, 4, 5, 6, 7, 8]


def config_pd(replicas: int = 1024, record_capacity: int = 1 << 15) -> List[Job]:
    """Decode-only p630d20 at 9 rates: WAIT with the fluid thresholds, then
    FCFS with a 1 % admission reserve (the decode-only baseline), on the same
    replica streams."""
    jobs = []
    for pol in ("wait", "fcfs"):
        for lam, n in zip(PD_RATES, PD_THRESHOLDS):
            wl = Workload(prompt_len=[PD_CONTEXT], lam=[lam], d0=10.0, d1=5e-5, C=137000,
                          policy=pol, n=[n] if pol == "wait" else [],
                          out_len=[PD_DECODE - 1], reserve=0.01 if pol == "fcfs" else 0.0,
                          hist_edges=default_edges(10.0), record_capacity=record_capacity)
            jobs.append(Job(wl, 0, ids(replicas)))
    return jobs


# ------------------------------------------------- time-varying rates ----


def diurnal_profile(m: int, span: float, points: int = 25, amp: float = 0.5,
                    cycles: float = 1.0, phases: Optional[Sequence[float]] = None):
    """Rate profile (rate_t [points], rate_f [m, points]) with
    f_j(t) = 1 + amp sin(2 pi cycles t / span + phase_j) at `points` equally
    spaced times over [0, span]; phases default to 2 pi j / m, so the type
    mix turns over the cycle as well as the total load."""
    t = np.linspace(0.0, span, points)
    if phases is None:
        phases = [2.0 * math.pi * j / m for j in range(m)]
    f = np.stack([1.0 + amp * np.sin(2.0 * math.pi * cycles * t / span + ph)
                  for ph in phases])
    return t, np.maximum(f, 0.0)


def with_profile(wl: Workload, rate_t, rate_f) -> Workload:
    return dataclasses.replace(wl, rate_t=np.asarray(rate_t, dtype=np.float64),
                               rate_f=np.asarray(rate_f, dtype=np.float64))


# Simulated time spanned by the cyclic workload's profile: 10^5 batches of the
# Llama-shaped WAIT mix near the fluid boundary cover about 6-9 x 10^8 ms.
TV_SPAN = 8.0e8


def config_cyclic(replicas: int = 1024, n_rates: int = 32, rate_index=None,
                  record_capacity: int = 1 << 15, span: float = TV_SPAN) -> List[Job]:
    """config2's WAIT jobs with time-varying rates: type j arrives at
    lam_j (1 + 0.5 sin(4 pi t / span + 2 pi j / 3)), two cycles over [0, span],
    piecewise linear through 25 points."""
    rt, rf = diurnal_profile(3, span, points=25, cycles=2.0)
    return [Job(with_profile(j.wl, rt, rf), j.seed, j.replica_ids)
            for j in config2(replicas, n_rates, rate_index, record_capacity)]


# ------------------------------------------------------------- traces ----


def trace_workload(policy: str, prompt_len, out_len, d0, d1, C, n, times, types,
                   lengths=None, seg_end=None, reserve=0.0, out_cap=0,
                   record_capacity=1 << 12, stage_caps=None) -> Workload:
    """Workload whose arrivals are the given (time, type[, length]) list."""
    times = np.asarray(times, dtype=np.float64)
    types = np.asarray(types, dtype=np.int32)
    if lengths is None:
        lengths = np.asarray([out_len[t] for t in types], dtype=np.int32)
    lengths = np.asarray(lengths, dtype=np.int32)
    return Workload(prompt_len=list(prompt_len), lam=[0.0] * len(prompt_len),
                    d0=d0, d1=d1, C=C, policy=policy, n=list(n),
                    out_len=None if out_len is None else list(out_len),
                    out_cap=out_cap, seg_end=seg_end, reserve=reserve,
                    hist_edges=default_edges(d0, 64),
                    record_capacity=record_capacity,
                    trace=(times, types, lengths),
                    stage_caps=None if stage_caps is None else list(stage_caps))
