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
* segment-design memory bound (Section 5.2 and the appendix on the
  segment-wise design): ``segment_design`` (delta_k, sbar_k), ``base_memory``
  (M^pi), ``theta_root``, ``memory_requirement`` (M^pi, the deterministic
  boundary term, the logarithmic buffer), ``fluid_segment_thresholds``,
  ``equal_rate_cuts`` and ``memory_vs_segments`` (the decomposition against L).
* time-varying rates (appendix, time-varying arrival rates): expected window
  arrivals ``window_arrivals``, the worst window load ``window_load_sup``
  (Lambda^pi), worst continuation probabilities ``continuation_sup`` (p*_k),
  the time-averaged fluid throughput ``fluid_throughput_tv``, a full batch's
  duration ``full_batch_time`` and the threshold conditions
  ``check_time_varying``.
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


# ------------------------------------------------- time-varying rates ----
# Intensities lam_j f_j(t), f_j linear between the profile points rate_t and
# constant outside them (the simulator's rate profile).  The appendix on
# time-varying rates replaces constant-rate threshold conditions by conditions
# on the expected arrivals in service windows:
#   A_j(t, h) = zeta * integral_t^{min(T, t + h / zeta)} lam_j^u du,
#   Lambda^pi = sup_t sum_j A_j(t, Delta^pi) < n_1,
#   p_k^* = sup over windows of sum_{r >= k} A_r / sum_{r >= k-1} A_r
#         < n_k / n_{k-1},
# and benchmarks throughput by (1/T) integral_0^T sum_j lam_j^t l'_j dt.


def _pl(rate_t, vals, t):
    """Piecewise-linear profile value(s) at t (constant outside)."""
    return np.interp(t, rate_t, vals)


def _pl_integral(rate_t, vals, a: float, b: float) -> float:
    """Exact integral over [a, b] (a <= b) of a piecewise-linear profile."""
    if not b > a:
        return 0.0
    inner = [x for x in rate_t if a < x < b]
    pts = np.array([a, *inner, b], dtype=np.float64)
    v = _pl(rate_t, vals, pts)
    return float(np.sum(np.diff(pts) * (v[1:] + v[:-1]) / 2.0))


def profile_intensities(lam: Sequence[float], rate_t, rate_f) -> np.ndarray:
    """lam_j f_j at the profile points, [m][P]."""
    f = np.asarray(rate_f, dtype=np.float64).reshape(len(lam), len(rate_t))
    return np.asarray(lam, dtype=np.float64)[:, None] * f


def window_arrivals(lam, rate_t, rate_f, t: float, h: float, zeta: float = 1.0,
                    T: float = math.inf) -> np.ndarray:
    """A_j(t, h) for every type j."""
    rt = np.asarray(rate_t, dtype=np.float64)
    inten = profile_intensities(lam, rt, rate_f)
    b = min(T, t + h / zeta)
    return np.array([zeta * _pl_integral(rt, row, t, b) for row in inten])


def window_load_sup(lam, rate_t, rate_f, h: float, T: float, zeta: float = 1.0):
    """(Lambda, t*): the largest total expected arrivals sum_j A_j(t, h) over
    window starts t in [0, T], and a start attaining it.  Exact: the window
    integral is piecewise quadratic in t, its breakpoints are the profile
    points, the points minus the window length and T minus it; the maximum
    lies at a breakpoint or where the derivative (linear between breakpoints)
    vanishes."""
    rt = np.asarray(rate_t, dtype=np.float64)
    tot = profile_intensities(lam, rt, rate_f).sum(axis=0)
    w = h / zeta

    def g(t):
        return zeta * _pl_integral(rt, tot, t, min(T, t + w))

    def dg(t, side):
        # one-sided derivative of g at t (side = +1 right, -1 left)
        e = side * 1e-12 * max(1.0, abs(t), w)
        up = _pl(rt, tot, t + w) if t + e + w < T else 0.0
        return zeta * (up - _pl(rt, tot, t))

    cand = {0.0, float(T)}
    for x in list(rt) + list(rt - w) + [T - w]:
        if 0.0 <= x <= T:
            cand.add(float(x))
    pts = sorted(cand)
    roots = []
    for a, b in zip(pts[:-1], pts[1:]):
        da, db = dg(a, +1), dg(b, -1)
        if da > 0 > db:
            roots.append(a + (b - a) * da / (da - db))
    best = max(pts + roots, key=g)
    return g(best), best


def _ratio_sup(num, den, rate_t, T):
    """sup over t in [0, T] with den(t) > 0 of num(t) / den(t), num and den
    piecewise linear on the same points (0 <= num <= den).  On each piece the
    ratio of two linear functions is monotone, so the supremum is at a piece
    end, or a one-sided limit where den vanishes (ratio of the slopes)."""
    rt = np.asarray(rate_t, dtype=np.float64)
    pts = sorted({0.0, float(T), *[float(x) for x in rt if 0.0 < x < T]})
    best = 0.0
    for a, b in zip(pts[:-1], pts[1:]):
        na, nb = _pl(rt, num, a), _pl(rt, num, b)
        da, db = _pl(rt, den, a), _pl(rt, den, b)
        if da <= 0.0 and db <= 0.0:
            continue
        for n_end, d_end in ((na, da), (nb, db)):
            if d_end > 0.0:
                best = max(best, n_end / d_end)
            else:  # den -> 0 at this end: the limit is the ratio of slopes
                best = max(best, (nb - na) / (db - da))
    if len(pts) == 1 and _pl(rt, den, 0.0) > 0.0:  # T = 0: the single instant
        best = _pl(rt, num, 0.0) / _pl(rt, den, 0.0)
    return best


def segment_intensities(lam, rate_t, rate_f, seg_end: Sequence[int],
                        out_len: Optional[Sequence[int]] = None,
                        cdf: Optional[np.ndarray] = None, cap: int = 0) -> np.ndarray:
    """Intensity of requests whose final output length lies in each segment,
    at the profile points, [L][P]."""
    inten = profile_intensities(lam, rate_t, rate_f)
    out = np.zeros((len(seg_end), len(rate_t)))
    for j in range(len(lam)):
        unit = [0.0] * len(lam)
        unit[j] = 1.0
        share = segment_rates(unit, seg_end, out_len=out_len, cdf=cdf, cap=cap)
        out += np.outer(share, inten[j])
    return out


def continuation_sup(seg_inten: np.ndarray, rate_t, T: float) -> list:
    """p*_k for k = 1..L-1 (the probability that a request reaching the end
    of segment k goes on, at its worst over [0, T]): the supremum of the
    instantaneous ratio sum_{r > k} / sum_{r >= k} of segment intensities,
    which bounds the ratio over any window (a weighted average of it) and is
    approached by short windows."""
    S = np.asarray(seg_inten, dtype=np.float64)
    return [_ratio_sup(S[k + 1:].sum(axis=0), S[k:].sum(axis=0), rate_t, T)
            for k in range(S.shape[0] - 1)]


def fluid_throughput_tv(lam, rate_t, rate_f, out_len: Sequence[float], T: float) -> float:
    """(1/T) integral_0^T sum_j lam_j^t l'_j dt (decode tokens per unit time)."""
    rt = np.asarray(rate_t, dtype=np.float64)
    inten = profile_intensities(lam, rt, rate_f)
    return float(sum(lp * _pl_integral(rt, row, 0.0, T)
                     for lp, row in zip(out_len, inten)) / T)


def full_batch_time(d0: float, d1: float, prompt_len: float, seg_end: Sequence[int],
                    n: Sequence[float]) -> float:
    """Duration of a batch holding n_k prompts at every stage of segment k:
    segment 1 spans stages 0..r_1 (prefill charges l, stage s charges l + s),
    segment k the stages r_{k-1}+1..r_k."""
    tokens, lo = 0.0, 0
    for k, (r, nk) in enumerate(zip(seg_end, n)):
        stages = range(lo, r + 1)
        tokens += nk * sum(prompt_len + s for s in stages)
        lo = r + 1
    return d0 + d1 * tokens


def check_time_varying(lam, rate_t, rate_f, n: Sequence[float], delta: float, T: float,
                       seg_inten: Optional[np.ndarray] = None, zeta: float = 1.0) -> dict:
    """The threshold conditions for time-varying rates: Lambda^pi < n_1 with
    Lambda^pi the worst expected arrivals in a window of length delta (a full
    batch's service time), and p*_k < n_{k+1} / n_k at every boundary (when
    segment intensities are given)."""
    Lam, t_star = window_load_sup(lam, rate_t, rate_f, delta, T, zeta)
    out = {"Lambda_pi": Lam, "t_star": t_star, "load_ok": Lam < n[0]}
    if seg_inten is not None:
        p = continuation_sup(seg_inten, rate_t, T)
        out["p_star"] = p
        out["continuation_ok"] = all(pk < n[k + 1] / n[k] for k, pk in enumerate(p))
    return out


# ------------------------------------------- segment-design memory bound ----
# Nested WAIT over L segments with boundaries r_1 < ... < r_L (Section 5.2 and
# the appendix on the segment-wise design): delta_1 = r_1 + 1, sbar_1 = r_1 / 2,
# delta_k = r_k - r_{k-1}, sbar_k = (r_{k-1} + 1 + r_k) / 2 for k >= 2;
#   M^pi = sum_k n_k (lbar_k + sbar_k) delta_k,
#   M_req = M^pi + sum_{k>=2} (lbar_k + r_{k-1}) n_k
#         + sum_{k>=2} (lbar_k + r_{k-1}) / theta_k * ln(m (1 + zeta T / d0) / delta),
# theta_k > 0 solving exp(-theta n_k) (1 - p_k + p_k e^theta)^{n_{k-1}} = 1.


def segment_design(seg_end: Sequence[int]) -> list:
    """(delta_k, sbar_k) per segment."""
    out, prev = [], 0
    for k, r in enumerate(seg_end):
        out.append((r + 1, r / 2.0) if k == 0 else (r - prev, (prev + 1 + r) / 2.0))
        prev = r
    return out


def _per_segment(l_bar, L):
    return list(l_bar) if isinstance(l_bar, (list, tuple, np.ndarray)) else [l_bar] * L


def base_memory(n: Sequence[float], seg_end: Sequence[int], l_bar) -> float:
    """M^pi, with a common prompt length or per-segment envelopes lbar_k."""
    lb = _per_segment(l_bar, len(seg_end))
    return float(sum(nk * (lk + sb) * dk
                     for nk, lk, (dk, sb) in zip(n, lb, segment_design(seg_end))))


def theta_root(n_k: float, n_prev: float, p_k: float) -> float:
    """The positive root of h(theta) = n_prev ln(1 - p + p e^theta) - theta n_k
    (h(0) = 0, h'(0) = n_prev p - n_k < 0, h convex and eventually
    increasing), found by bracketing and Brent's method."""
    from scipy.optimize import brentq
    if not (0.0 < p_k < 1.0 and n_prev * p_k < n_k):
        raise ValueError("theta_k needs 0 < p_k < 1 and n_{k-1} p_k < n_k")

    def h(th):
        # ln(1 - p + p e^th) = th + ln(p + (1 - p) e^-th), stable for large th
        return n_prev * (th + math.log(p_k + (1.0 - p_k) * math.exp(-th))) - th * n_k

    a = 1e-9 * max(1.0, 1.0 / n_k)
    while h(a) >= 0.0:   # step inside the negative region right of 0
        a *= 0.5
    b = 1.0
    while h(b) <= 0.0:
        b *= 2.0
    return float(brentq(h, a, b, xtol=1e-15, rtol=1e-15, maxiter=500))


def memory_requirement(n: Sequence[float], seg_end: Sequence[int], l_bar,
                       p: Sequence[float], m: int, zeta_T: float, d0: float,
                       delta: float) -> dict:
    """The three terms of the segment-design memory bound and their sum;
    p[k-1] is the continuation probability into segment k + 1 (k = 1..L-1)."""
    L = len(seg_end)
    lb = _per_segment(l_bar, L)
    term1 = base_memory(n, seg_end, lb)
    log_term = math.log(m * (1.0 + zeta_T / d0) / delta)
    term2 = term3 = 0.0
    thetas = []
    for k in range(1, L):
        th = theta_root(n[k], n[k - 1], p[k - 1])
        thetas.append(th)
        w = lb[k] + seg_end[k - 1]
        term2 += w * n[k]
        term3 += w * log_term / th
    return {"term1": term1, "term2": term2, "term3": term3,
            "total": term1 + term2 + term3, "theta": thetas}


def fluid_segment_thresholds(seg_rates: Sequence[float], seg_end: Sequence[int], l_bar,
                             d0: float, d1: float, eta: float = 0.05,
                             slack: float = 0.05) -> Optional[list]:
    """Thresholds meeting the segment-design conditions: n_k = n_1 prod_{r<k} q_r
    with q_k = min(p_k + eta, 0.99) (so p_k < n_k / n_{k-1} < 1), and n_1 a
    factor (1 + slack) above the smallest value with
    d0 + d1 M^pi(n) < n_1 / sum_k lam'_k.  None when no n_1 satisfies it
    (d1 M^pi per unit n_1 at least 1 / sum lam')."""
    p = continuation_probabilities(seg_rates)
    rel = [1.0]
    for x in p:
        rel.append(rel[-1] * min(x + eta, 0.99))
    S = base_memory(rel, seg_end, l_bar)        # M^pi per unit n_1
    gap = 1.0 / sum(seg_rates) - d1 * S
    if gap <= 0.0:
        return None
    n1 = (1.0 + slack) * d0 / gap
    return [n1 * r for r in rel]


def equal_rate_cuts(out_len: Sequence[int], rates: Sequence[float], L: int) -> list:
    """Segment boundaries for L segments over output-length classes sorted by
    length: cut after the class where the cumulative arrival rate first reaches
    k / L of the total (each boundary a class's output length, strictly
    increasing; fewer than L segments if classes are too coarse)."""
    order = np.argsort(out_len)
    lens = np.asarray(out_len)[order]
    cum = np.cumsum(np.asarray(rates, dtype=np.float64)[order])
    cuts = []
    for k in range(1, L):
        i = int(np.searchsorted(cum, k / L * cum[-1] * (1 - 1e-12)))
        r = int(lens[min(i, len(lens) - 1)])
        if (not cuts or r > cuts[-1]) and r < lens[-1]:
            cuts.append(r)
    return cuts + [int(lens[-1])]


def memory_vs_segments(prompt_len: float, out_len: Sequence[int], rates: Sequence[float],
                       L_values: Sequence[int], d0: float, d1: float, zeta_T: float,
                       delta: float, eta: float = 0.05, slack: float = 0.05) -> list:
    """The decomposition of the memory bound against the number of segments L
    (common prompt length): for each L, equal-rate cuts, fluid thresholds and
    the three terms.  Rows with infeasible thresholds are omitted."""
    rows = []
    for L in L_values:
        seg_end = equal_rate_cuts(out_len, rates, L)
        seg_rates = segment_rates(rates, seg_end, out_len=out_len)
        n = fluid_segment_thresholds(seg_rates, seg_end, prompt_len, d0, d1, eta, slack)
        if n is None:
            continue
        p = continuation_probabilities(seg_rates)
        mr = memory_requirement(n, seg_end, prompt_len, p, len(out_len), zeta_T, d0, delta)
        rows.append({"L": len(seg_end), "seg_end": seg_end, "n": n, **mr})
    return rows
