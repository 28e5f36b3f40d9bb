"""Fluid-equilibrium and threshold calculator (test infrastructure).

Closed forms of arXiv 2504.11320 used as checks on the simulator and to derive
workload parameters.  Only tests, the smoke check and the benchmark's CPU
baseline may import this module; the GPU path never does.

Sections followed:
  * Section 3.1, single-type fluid model: n* = d0 lam / (1 - d1 lam (l'+1)(l+l'/2)),
    eq. (memory_single), eq. (throughput_fluid);
  * Section 3.2, multi-type fluid model: A = sum_j lam_j (l'_j+1)(l_j+l'_j/2),
    eq. (memory_multi2) M* = d0 A / (1 - d1 A), eq. (time_fluid)
    dT* = d0 / (1 - d1 A), n_j* = lam_j dT*, eq. (throughput_fluid_multiple);
  * Proposition 1: instability when d1 A >= 1 (single type: lam d1 (l'+1)(l+l'/2) >= 1);
  * Section 4.3, eq. (wait_thresholds): M^pi = sum_j n_j (l'_j+1)(l_j+l'_j/2)
    and d0 + d1 M^pi <= n_j / lam_j;
  * Section 5.2 and Appendix A (segment design): delta_1 = r_1+1,
    sbar_1 = r_1/2, delta_k = r_k - r_{k-1}, sbar_k = (r_{k-1}+1+r_k)/2,
    M^pi = sum_k n_k (l + sbar_k) delta_k, eq. (nested_wait_thresholds_L),
    eq. (nested_wait_memory_L) with theta_k the positive root of
    exp(-theta n_k) (1 - p_k + p_k e^theta)^{n_{k-1}} = 1;
  * Section 6 (WAIT and Nested WAIT settings): threshold calibration from a
    system cap tl, q_k = min(p_k + eta, 0.99), n_k = n_1 prod_{r<k} q_r,
    sum_k dl_k n_k = tl, segment caps B_k = dl_k n_k.
"""
from __future__ import annotations

import math
from typing import Sequence


def stage_work(l: float, lp: float) -> float:
    """(l'+1)(l+l'/2): total cached tokens a prompt carries over its l'+1
    processing stages (Section 3.1)."""
    return (lp + 1.0) * (l + lp / 2.0)


def single_type(l: float, lp: float, lam: float, d0: float, d1: float) -> dict:
    """Section 3.1: n*, M*, throughput*; None entries when Prop. 1 applies."""
    w = stage_work(l, lp)
    denom = 1.0 - d1 * lam * w
    if denom <= 0.0:
        return {"stable": False, "nstar": math.inf, "Mstar": math.inf,
                "throughput": lam * lp}
    nstar = d0 * lam / denom
    return {"stable": True, "nstar": nstar, "Mstar": nstar * w,
            "throughput": lam * lp}


def load_A(l: Sequence[float], lp: Sequence[float], lam: Sequence[float]) -> float:
    """A = sum_j lam_j (l'_j+1)(l_j+l'_j/2) (Section 3.2)."""
    return sum(x * stage_work(a, b) for a, b, x in zip(l, lp, lam))


def fluid(l, lp, lam, d0: float, d1: float) -> dict:
    """Section 3.2 multi-type fluid equilibrium."""
    A = load_A(l, lp, lam)
    thr = sum(x * b for b, x in zip(lp, lam))
    if d1 * A >= 1.0:
        return {"A": A, "stable": False, "Mstar": math.inf, "dTstar": math.inf,
                "nstar": [math.inf] * len(lam), "throughput": thr}
    dT = d0 / (1.0 - d1 * A)
    return {"A": A, "stable": True, "Mstar": d0 * A / (1.0 - d1 * A),
            "dTstar": dT, "nstar": [x * dT for x in lam], "throughput": thr}


def fluid_mean_work(ES: float, Lam: float, d0: float, d1: float) -> float:
    """M* for a mix with mean stage work E[S] at total rate Lam:
    A = Lam E[S] (Section 3.2, with lam_j = pi_j Lam)."""
    A = Lam * ES
    return d0 * A / (1.0 - d1 * A) if d1 * A < 1.0 else math.inf


def lambda_star(ES: float, d0: float, d1: float, C: float) -> float:
    """Total rate at which the fluid memory requirement equals C:
    d0 A / (1 - d1 A) = C  <=>  A = C / (d0 + d1 C), A = Lam E[S]."""
    return C / ((d0 + d1 * C) * ES)


# ----------------------------------------------------------------- WAIT ----

def wait_mpi(n, l, lp) -> float:
    """M^pi of eq. (wait_thresholds)."""
    return sum(nj * stage_work(a, b) for nj, a, b in zip(n, l, lp))


def wait_conditions(n, l, lp, lam, d0, d1, C) -> dict:
    """The three lines of eq. (wait_thresholds)."""
    mpi = wait_mpi(n, l, lp)
    dT = d0 + d1 * mpi
    tol = 1e-12  # relative slack for rounding in the closed forms
    balance = all(dT <= (nj / x) * (1 + tol) for nj, x in zip(n, lam) if x > 0)
    fl = fluid(l, lp, lam, d0, d1)
    memory = fl["Mstar"] <= mpi * (1 + tol) and mpi <= C
    return {"Mpi": mpi, "dT": dT, "balance": balance,
            "Mstar": fl["Mstar"], "memory": memory, "holds": balance and memory}


def wait_thresholds_from_fluid(l, lp, lam, d0, d1) -> list[int]:
    """Integer thresholds n_j = max(1, ceil(n_j*)) where the fluid equilibrium
    exists, else 1."""
    fl = fluid(l, lp, lam, d0, d1)
    if not fl["stable"]:
        return [1] * len(lam)
    return [max(1, math.ceil(x - 1e-12)) for x in fl["nstar"]]


# --------------------------------------------------------------- Nested ----

def seg_delta_sbar(seg_end: Sequence[int]):
    """delta_k and sbar_k of the segment design (Appendix A)."""
    out = []
    prev = 0
    for k, r in enumerate(seg_end):
        if k == 0:
            out.append((r + 1, r / 2.0))
        else:
            out.append((r - prev, (prev + 1 + r) / 2.0))
        prev = r
    return out


def nested_mpi(n, seg_end, l_env) -> float:
    """M^pi = sum_k n_k (lbar_k + sbar_k) delta_k; l_env is a common prefill
    length or the per-segment envelope lbar_k."""
    if not isinstance(l_env, (list, tuple)):
        l_env = [l_env] * len(seg_end)
    return sum(nk * (lk + sb) * dk
               for nk, lk, (dk, sb) in zip(n, l_env, seg_delta_sbar(seg_end)))


def continuation_probs(seg_rates: Sequence[float]) -> list[float]:
    """p_k = lam'(k..L) / lam'(k-1..L) for k = 2..L (returned for k=2..L)."""
    tails = [sum(seg_rates[k:]) for k in range(len(seg_rates))]
    return [tails[k] / tails[k - 1] for k in range(1, len(seg_rates))]


def theta_root(n_k: float, n_km1: float, p_k: float) -> float:
    """Positive root of exp(-theta n_k)(1 - p + p e^theta)^{n_{k-1}} = 1,
    i.e. g(theta) = -theta n_k + n_{k-1} ln(1 - p + p e^theta) = 0, by
    bisection (requires n_{k-1} p < n_k and p > 0)."""
    if not (0.0 < p_k and n_km1 * p_k < n_k):
        raise ValueError("theta root needs 0 < p and n_{k-1} p < n_k")

    def g(th):
        # ln(1-p+p e^th) computed stably
        return -th * n_k + n_km1 * (th + math.log(p_k + (1.0 - p_k) * math.exp(-th)))

    lo, hi = 0.0, 1.0
    while g(hi) <= 0.0:
        hi *= 2.0
        if hi > 1e6:
            raise ValueError("no root")
    # g < 0 just right of 0 (derivative n_{k-1} p - n_k < 0)
    lo = hi * 1e-12
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if g(mid) > 0.0:
            hi = mid
        else:
            lo = mid
    return 0.5 * (lo + hi)


def nested_m_req(n, seg_end, l_env, p, m: int, zeta_T: float, d0: float,
                 delta: float) -> dict:
    """eq. (nested_wait_memory_L): base term, deterministic boundary term and
    the logarithmic safety buffer."""
    L = len(seg_end)
    if not isinstance(l_env, (list, tuple)):
        l_env = [l_env] * L
    base = nested_mpi(n, seg_end, l_env)
    term2 = 0.0
    term3 = 0.0
    logt = math.log(m * (1.0 + zeta_T / d0) / delta)
    thetas = []
    for k in range(1, L):
        th = theta_root(n[k], n[k - 1], p[k - 1])
        thetas.append(th)
        w = l_env[k] + seg_end[k - 1]
        term2 += w * n[k]
        term3 += w * logt / th
    return {"Mpi": base, "term2": term2, "term3": term3,
            "Mreq": base + term2 + term3, "theta": thetas}


def calibrate(tl: float, widths: Sequence[int], p: Sequence[float],
              eta: float) -> dict:
    """Section 6 threshold calibration: q_k = min(p_k + eta, 0.99),
    n_k = n_1 prod_{r<k} q_r, sum_k widths_k n_k = tl, B_k = widths_k n_k."""
    q = [min(x + eta, 0.99) for x in p]
    rel = [1.0]
    for x in q:
        rel.append(rel[-1] * x)
    n1 = tl / sum(w * r for w, r in zip(widths, rel))
    n = [n1 * r for r in rel]
    B = [w * x for w, x in zip(widths, n)]
    return {"n": n, "B": B}
