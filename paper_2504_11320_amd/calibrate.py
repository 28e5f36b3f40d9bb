"""Fluid quantities and threshold calibration for setting up simulations
(arXiv 2504.11320).  Host-side helpers of the simulator's API.

* ``stage_work`` / ``mean_stage_work``: the tokens a request holds summed over
  its processing stages, S = sum_{s=0}^{L} (l + s) = (L + 1)(l + L / 2)
  (Section 3.1), and its mean over a type mix and output-length law.
* ``fluid_boundary``: the total arrival rate at which the fluid memory
  requirement M* = d0 A / (1 - d1 A), A = Lambda E[S] (Section 3.2), equals the
  KV budget C: Lambda* = C / ((d0 + d1 C) E[S]).
* ``length_pmf``: P(L = s) of the output-length law encoded as the library's
  u32 CDF table (L is the smallest s with w < T[s], else the cap).
* ``segment_rates`` / ``continuation_probabilities``: the arrival rate of
  requests whose final output length falls in each Nested WAIT segment, and
  p_k = (sum_{r > k} rate_r) / (sum_{r >= k} rate_r) (Section 6).
* ``calibrate_nested`` / ``calibrate_wait``: the Section 6 allocation of a
  system-wide batch-size cap tl to per-stage thresholds.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np


def stage_work(l: float, L: float) -> float:
    """Sum over the L + 1 processing stages of the tokens held: (L+1)(l+L/2)."""
    return (L + 1.0) * (l + L / 2.0)


def length_pmf(cdf_row: Sequence[int], cap: int) -> np.ndarray:
    """P(L = s) for s = 0..cap (entry 0 is 0) from a u32 CDF table of
    cap - 1 thresholds T[1..cap-1]: P(L = s) = (T[s] - T[s-1]) / 2^32 with
    T[0] = 0 and T[cap] = 2^32."""
    t = np.concatenate(([0.0], np.asarray(cdf_row, dtype=np.float64), [2.0 ** 32]))
    if len(t) != cap + 1:
        raise ValueError("a CDF row holds cap - 1 thresholds")
    pmf = np.zeros(cap + 1)
    pmf[1:] = np.diff(t) / 2.0 ** 32
    return pmf


def mean_stage_work(prompt_len: Sequence[int], mix: Sequence[float],
                    out_len: Optional[Sequence[int]] = None,
                    cdf: Optional[np.ndarray] = None, cap: int = 0) -> float:
    """E[S] over a type mix (weights summing to 1) with known output lengths
    ``out_len`` or the CDF tables ``cdf`` [m][cap - 1]."""
    total = 0.0
    for j, (l, w) in enumerate(zip(prompt_len, mix)):
        if out_len is not None:
            total += w * stage_work(l, out_len[j])
        else:
            pmf = length_pmf(cdf[j], cap)
            s = np.arange(cap + 1, dtype=np.float64)
            total += w * float(np.sum(pmf * (s + 1.0) * (l + s / 2.0)))
    return total


def fluid_boundary(mean_work: float, d0: float, d1: float, C: float) -> float:
    """Lambda* (requests per unit time) at which M* = C."""
    return C / ((d0 + d1 * C) * mean_work)


def segment_rates(lam: Sequence[float], seg_end: Sequence[int],
                  out_len: Optional[Sequence[int]] = None,
                  cdf: Optional[np.ndarray] = None, cap: int = 0) -> list:
    """Rate of requests whose final output length lies in (r_{k-1}, r_k]."""
    rates = [0.0] * len(seg_end)
    bounds = [0] + list(seg_end)
    for j, x in enumerate(lam):
        if out_len is not None:
            for k in range(len(seg_end)):
                if bounds[k] < out_len[j] <= bounds[k + 1]:
                    rates[k] += x
        else:
            pmf = length_pmf(cdf[j], cap)
            for k in range(len(seg_end)):
                rates[k] += x * float(np.sum(pmf[bounds[k] + 1: bounds[k + 1] + 1]))
    return rates


def continuation_probabilities(seg_rates: Sequence[float]) -> list:
    """p_k for k = 1..L-1: the probability that a request in segment k goes
    on to segment k + 1."""
    out = []
    for k in range(len(seg_rates) - 1):
        here = sum(seg_rates[k:])
        out.append(sum(seg_rates[k + 1:]) / here if here > 0 else 0.0)
    return out


def _spread(total: int, stages: int) -> list:
    """An integer total over ``stages`` stages as evenly as possible (the
    first ``total % stages`` stages take one more)."""
    base, extra = divmod(total, stages)
    return [base + 1] * extra + [base] * (stages - extra)


def calibrate_nested(tl: float, seg_end: Sequence[int], p: Sequence[float],
                     eta: float = 0.05) -> dict:
    """Section 6: q_k = min(p_k + eta, 0.99); n_k = n_1 prod_{r<k} q_r with
    n_1 solving sum_k dl_k n_k = tl, dl_k the number of decode stages of
    segment k (r_1, r_2 - r_1, ...); segment caps B_k = dl_k n_k rounded and
    spread as evenly as possible over the segment's stages.  ``thresholds`` is
    the per-segment threshold the simulator takes (one per segment):
    max(1, round(n_k))."""
    widths = [seg_end[0]] + [seg_end[k] - seg_end[k - 1] for k in range(1, len(seg_end))]
    if len(p) != len(seg_end) - 1:
        raise ValueError("one continuation probability per segment boundary")
    q = [min(x + eta, 0.99) for x in p]
    rel = [1.0]
    for x in q:
        rel.append(rel[-1] * x)
    n1 = tl / sum(w * r for w, r in zip(widths, rel))
    n = [n1 * r for r in rel]
    caps = [int(round(w * x)) for w, x in zip(widths, n)]
    return {"n": n, "segment_caps": caps,
            "stage_caps": [_spread(c, w) for c, w in zip(caps, widths)],
            "thresholds": [max(1, int(round(x))) for x in n]}


def calibrate_wait(tl: int, out_len: int) -> dict:
    """Section 6, single type: the cap tl spread over the prefill and l'
    decode stages; ``threshold`` is the uniform per-stage threshold the
    simulator takes, max(1, floor(tl / (l' + 1)))."""
    stages = out_len + 1
    return {"stage_caps": _spread(int(tl), stages),
            "threshold": max(1, int(tl) // stages)}
