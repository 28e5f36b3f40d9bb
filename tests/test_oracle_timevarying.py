"""Pins of the oracle's time-varying arrivals (the paper's appendix on
time-varying rates: independent nonhomogeneous Poisson processes with
continuous bounded intensities lambda_j^t).  Type j arrives at intensity
lam_j f_j(t), f_j piecewise linear through the profile points and constant
outside them, sampled by thinning a Poisson process at rate lam_j max f_j.

What fixes the answer independently of the oracle's code:
* a constant profile is a homogeneous Poisson process at lam_j * c (its draws
  are then the homogeneous ones, bit for bit);
* arrival counts in a window are Poisson with mean lam_j * integral of f_j
  over the window (the integral of a piecewise-linear function is exact by
  the trapezoid rule), tested over many replicas;
* no arrival falls where the intensity is zero, and an intensity that ends at
  zero gives finitely many arrivals, Poisson with mean lam_j * total integral;
* accepted arrivals are a subset of the candidate process: the arrival with
  Philox counter k sits at the k-th candidate time of the homogeneous process
  at the bound and carries that candidate's output length.
"""
import math

import numpy as np
import pytest

import workloads as W
from tests.parity_util import compare


def _wl(policy="wait", lam=(0.05, 0.02), rate_t=None, rate_f=None, m=2, C=4000,
        out_len=(8, 24), n=(2, 1)):
    return W.Workload(prompt_len=[16, 64][:m], lam=list(lam[:m]), d0=5.0, d1=0.01,
                      C=C, policy=policy, n=list(n[:m]), out_len=list(out_len[:m]),
                      hist_edges=W.default_edges(5.0, 64), record_capacity=1 << 14,
                      rate_t=None if rate_t is None else np.asarray(rate_t, float),
                      rate_f=None if rate_f is None else np.asarray(rate_f, float))


def _integral(rate_t, f, a, b):
    """Integral over [a, b] of the piecewise-linear f (constant outside)."""
    pts = sorted({a, b, *[t for t in rate_t if a < t < b]})
    vals = np.interp(pts, rate_t, f)
    return float(sum((pts[i + 1] - pts[i]) * (vals[i] + vals[i + 1]) / 2.0
                     for i in range(len(pts) - 1)))


def test_constant_profile_is_homogeneous(oracle_lib):
    """f_j = c_j everywhere: bit-identical to rates lam_j * c_j, for every
    policy, through the whole simulation."""
    from oracle import oracle as O
    c = [1.5, 0.25]
    lam = (0.05, 0.02)
    for pol, n in (("wait", (2, 1)), ("fcfs", ()), ("nested", (2, 1))):
        kw = dict(policy=pol, n=n)
        if pol == "nested":
            kw["n"] = (2, 1)
        tv = _wl(lam=lam, rate_t=[0.0, 100.0, 7000.0],
                 rate_f=[[c[0]] * 3, [c[1]] * 3], **kw)
        hom = _wl(lam=(lam[0] * c[0], lam[1] * c[1]), **kw)
        if pol == "nested":
            tv.seg_end = hom.seg_end = [8, 24]
        a = O.run_job(W.Job(tv, 11, W.ids(4)), 1500)
        b = O.run_job(W.Job(hom, 11, W.ids(4)), 1500)
        for f in O.INT_FIELDS + O.F64_FIELDS:
            assert np.array_equal(a[f], b[f]), (pol, f)
        assert np.array_equal(a["hist"], b["hist"])
        assert a["arrivals"].min() > 100


def test_arrivals_sit_on_candidates(oracle_lib):
    """With f_j > 0 everywhere, arrival a with counter k is the k-th candidate
    of the homogeneous process at lam_j max f_j: same time, same length."""
    from oracle import oracle as O
    rt = [0.0, 500.0, 1000.0, 2000.0]
    rf = [[1.0, 0.2, 2.0, 0.5], [0.1, 0.1, 0.4, 0.05]]
    cdf = np.stack([W.geometric_cdf_table(6.0, 32), W.geometric_cdf_table(12.0, 32)])
    tv = W.Workload(prompt_len=[16, 64], lam=[0.05, 0.3], d0=5.0, d1=0.01, C=4000,
                    policy="wait", n=[2, 1], out_cap=32, out_cdf=cdf,
                    rate_t=np.array(rt), rate_f=np.array(rf))
    for j in range(2):
        fmax = max(rf[j])
        hom = W.Workload(prompt_len=[16, 64], lam=[0.05 * max(rf[0]), 0.3 * max(rf[1])],
                         d0=5.0, d1=0.01, C=4000, policy="wait", n=[2, 1], out_cap=32,
                         out_cdf=cdf)
        t, L, k, fl = O.arrival_times(tv, 5, 3, j, 200)
        th, Lh, kh, _ = O.arrival_times(hom, 5, 3, j, int(k.max()) + 1)
        assert fl == 0
        assert np.array_equal(kh, np.arange(len(kh)))
        assert np.all(np.diff(k.astype(np.int64)) >= 1)
        assert np.array_equal(t, th[k]) and np.array_equal(L, Lh[k])
        # the acceptance fraction follows the mean of f / fmax over the span
        span = float(t[-1])
        frac = _integral(rt, rf[j], 0.0, span) / (fmax * span)
        n_cand = int(k[-1]) + 1
        sd = math.sqrt(frac * (1 - frac) / n_cand)
        assert abs(len(t) / n_cand - frac) < 5 * sd + 0.01


def test_window_counts_follow_integral(oracle_lib):
    """Counts per window over 4000 replica streams: mean within 5 standard
    errors of lam * integral of f, variance near the mean (Poisson)."""
    from oracle import oracle as O
    rt = [0.0, 200.0, 400.0, 600.0, 1000.0]
    rf = [[0.5, 2.0, 2.0, 0.0, 1.0]]
    lam = 0.05
    wl = _wl(lam=(lam,), m=1, n=(1,), out_len=(4,), rate_t=rt, rate_f=rf)
    windows = [(0, 200), (200, 400), (400, 600), (550, 650), (600, 1000), (1000, 1400)]
    R = 4000
    counts = np.zeros((R, len(windows)))
    for r in range(R):
        t, _, _, _ = O.arrival_times(wl, 77, r, 0, 200)
        assert t[-1] > 1400
        for w, (a, b) in enumerate(windows):
            counts[r, w] = np.count_nonzero((t >= a) & (t < b))
    for w, (a, b) in enumerate(windows):
        mu = lam * _integral(rt, rf[0], a, b)
        mean = counts[:, w].mean()
        assert abs(mean - mu) < 5 * math.sqrt(mu / R), (a, b, mean, mu)
        var = counts[:, w].var(ddof=1)
        assert abs(var / mu - 1.0) < 0.15, (a, b, var, mu)


def test_zero_intensity(oracle_lib):
    """No arrival where f is zero; a profile ending at zero stops the type
    (time inf, no flag) after a Poisson number of arrivals."""
    from oracle import oracle as O
    rt = [0.0, 100.0, 200.0, 300.0, 400.0, 500.0]
    rf = [[0.0, 1.0, 0.0, 0.0, 1.0, 0.0]]
    lam = 0.1
    wl = _wl(lam=(lam,), m=1, n=(1,), out_len=(4,), rate_t=rt, rate_f=rf)
    tot = []
    for r in range(600):
        t, _, _, fl = O.arrival_times(wl, 9, r, 0, 400)
        assert fl == 0
        fin = t[np.isfinite(t)]
        assert np.all(np.isinf(t[len(fin):]))
        assert np.all((fin > 0) & (fin < 500))
        assert not np.any((fin >= 200) & (fin <= 300))
        tot.append(len(fin))
    mu = lam * _integral(rt, rf[0], 0.0, 500.0)  # 20
    assert abs(np.mean(tot) - mu) < 5 * math.sqrt(mu / len(tot))
    # a profile that starts at zero before its first point: nothing before it
    wl2 = _wl(lam=(lam,), m=1, n=(1,), out_len=(4,), rate_t=[50.0, 60.0],
              rate_f=[[0.0, 1.0]])
    t, _, _, _ = O.arrival_times(wl2, 9, 0, 0, 50)
    assert t[0] > 50.0
    # an all-zero profile never arrives; the simulation stalls at once
    wl3 = _wl(lam=(lam,), m=1, n=(1,), out_len=(4,), rate_t=[0.0], rate_f=[[0.0]])
    t, _, _, _ = O.arrival_times(wl3, 9, 0, 0, 3)
    assert np.all(np.isinf(t))
    r = O.run_one(wl3, 9, 0, 10)
    assert r["arrivals"] == 0 and r["flags"] == O.FLAG_STALL


def test_thinning_limit_flag(oracle_lib):
    """A positive intensity 2^-30 of its bound rejects 2^20 candidates in a
    row almost surely: the type stops and the flag says so."""
    from oracle import oracle as O
    wl = _wl(lam=(1.0,), m=1, n=(1,), out_len=(4,), rate_t=[0.0, 1.0],
             rate_f=[[1.0, 2.0 ** -30]])
    t, _, k, fl = O.arrival_times(wl, 4, 0, 0, 10)
    assert fl == O.FLAG_THIN_LIMIT
    assert np.isinf(t[-1])
    assert np.all(t[np.isfinite(t)] < 1.0 + 0.1)


def test_simulation_sees_the_profile(oracle_lib):
    """A WAIT run's request log holds exactly the merged per-type arrival
    streams up to its end time."""
    from oracle import oracle as O
    rt = [0.0, 300.0, 900.0]
    rf = [[0.2, 3.0, 1.0], [1.0, 0.0, 2.0]]
    wl = _wl(rate_t=rt, rate_f=rf)
    r = O.run_one(wl, 21, 6, 400, rlog_cap=4096)
    T = r["t_end"]
    streams = []
    for j in range(2):
        t, _, _, _ = O.arrival_times(wl, 21, 6, j, 4096)
        streams.append(t[t <= T])
    merged = np.sort(np.concatenate(streams))
    log = r["req_arr"][: r["arrivals"]]
    assert r["arrivals"] == len(merged) > 50
    assert np.array_equal(log, merged)


def test_integral_helper():
    """The trapezoid integral of a piecewise-linear profile (constant
    outside) against closed forms."""
    assert _integral([0.0, 1.0], [0.0, 2.0], 0.0, 1.0) == pytest.approx(1.0)
    assert _integral([0.0, 1.0], [0.0, 2.0], -1.0, 2.0) == pytest.approx(3.0)
    assert _integral([1.0, 3.0], [1.0, 1.0], 0.0, 10.0) == pytest.approx(10.0)
