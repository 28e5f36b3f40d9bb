"""Metrics derived from simulation results (arXiv 2504.11320, Section 2.4 and
the arrival-rate experiments of Section 6).  Host-side helpers of the
simulator's API: they read the per-replica result dictionary the binding
returns (``Simulation.results`` / ``run_batch``).

* ``summarize``: per-replica throughput (completed decode tokens per unit
  time), completion rate (completed requests per unit time; evicted prompts
  restart and are not completions), mean latency of completed requests, mean
  censored latency and TTFT (the areas divided by the arrivals), eviction and
  idle rates, peak memory.
* ``hist_percentile``: a latency percentile from a replica's histogram row
  (bin b holds latencies in [edge_{b-1}, edge_b)): the upper edge of the bin
  where the cumulative count reaches the quantile.
* ``job_means``: means and standard errors of a metric over each job's
  replicas.
* ``lambda_hat``: the stability point of a rate sweep, read as the largest
  tested rate up to which every rate's completion rate stays within a
  tolerance of its arrival rate.
* ``review_process``: a side simulator of the embedded review process of the
  critical threshold queue, for the identity E[W^B] = n E[B_stuck].
"""
from __future__ import annotations

from typing import Sequence

import numpy as np


def summarize(res: dict) -> dict:
    T = res["t_end"].astype(np.float64)
    done = res["completions"].astype(np.float64)
    arr = res["arrivals"].astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        return {
            "throughput_tokens": np.where(T > 0, res["completed_tokens"] / T, 0.0),
            "completion_rate": np.where(T > 0, done / T, 0.0),
            "mean_latency_completed": np.where(done > 0, res["lat_completed_sum"] / done,
                                               np.nan),
            "mean_latency_censored": np.where(arr > 0, res["lat_area"] / arr, np.nan),
            "mean_ttft_censored": np.where(arr > 0, res["ttft_area"] / arr, np.nan),
            "evictions_per_batch": np.where(res["batches"] > 0,
                                            res["evictions"] / res["batches"], 0.0),
            "busy_fraction": np.where(T > 0, res["busy_time"] / T, 0.0),
            "peak_mem": res["peak_mem"].astype(np.float64),
        }


def hist_percentile(hist_row: Sequence[int], edges: Sequence[float], q: float) -> float:
    """Upper edge of the bin holding the q-quantile (inf past the last edge,
    nan for an empty histogram)."""
    h = np.asarray(hist_row, dtype=np.float64)[: len(edges) + 1]
    total = h.sum()
    if total <= 0:
        return float("nan")
    b = int(np.searchsorted(np.cumsum(h), q * total, side="left"))
    return float(edges[b]) if b < len(edges) else float("inf")


def job_means(values: np.ndarray, counts: Sequence[int]) -> list:
    """(mean, standard error) of ``values`` over consecutive groups of
    ``counts`` replicas (the jobs of one launch, in order)."""
    out, start = [], 0
    for n in counts:
        v = np.asarray(values[start:start + n], dtype=np.float64)
        v = v[np.isfinite(v)]
        start += n
        if len(v) == 0:
            out.append((float("nan"), float("nan")))
            continue
        se = float(v.std(ddof=1) / np.sqrt(len(v))) if len(v) > 1 else float("nan")
        out.append((float(v.mean()), se))
    return out


def lambda_hat(rates: Sequence[float], completion_rates: Sequence[float],
               tol: float = 0.05) -> float:
    """Largest rate r_i such that completion_rate_k >= (1 - tol) r_k for every
    tested r_k <= r_i (0 if the lowest rate already falls short)."""
    order = np.argsort(np.asarray(rates, dtype=np.float64))
    best = 0.0
    for i in order:
        if completion_rates[i] >= (1.0 - tol) * rates[i]:
            best = float(rates[i])
        else:
            break
    return best


def review_process(n: int, B: int, reps: int, seed: int = 0) -> dict:
    """The embedded review process of the critical single-type threshold
    queue (the lemma on queue length and stuck time, Section 4.3): X^b ~
    Poisson(n) arrivals per review interval, W^{b+1} = W^b + X^b - n 1{W^b + X^b
    >= n}, W^0 = 0; a review is stuck when W^b + X^b < n.  Simulated for `reps`
    independent paths of B reviews (numpy, vectorised over paths).  Returns W^B,
    the stuck counts and the arrival totals per path."""
    rng = np.random.default_rng(seed)
    W = np.zeros(reps, dtype=np.int64)
    stuck = np.zeros(reps, dtype=np.int64)
    total = np.zeros(reps, dtype=np.int64)
    for _ in range(B):
        X = rng.poisson(n, reps)
        total += X
        s = W + X
        served = s >= n
        W = s - n * served
        stuck += ~served
    return {"W": W, "stuck": stuck, "arrivals": total}
