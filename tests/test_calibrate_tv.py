"""Pins of the host calculator for time-varying rates (the paper's appendix
on time-varying arrival rates: window loads A_j(t, h), their worst case
Lambda^pi, worst continuation probabilities p*_k, the time-averaged fluid
throughput).  Closed forms, reductions to the constant-rate formulas, and
brute force with numerical quadrature on random piecewise-linear profiles."""
import math

import numpy as np
import pytest
from scipy import integrate

from paper_2504_11320_amd import calibrate as K


def _rand_profile(rng, m, T, P):
    t = np.sort(rng.uniform(-0.1 * T, 1.1 * T, P))
    f = rng.uniform(0.0, 2.0, (m, P))
    f[rng.uniform(size=f.shape) < 0.25] = 0.0
    return t, f


def test_triangle_closed_form():
    """Peak H at t0, half-width a, window w <= 2a: the best window is centred
    on the peak and holds H w - H w^2 / (4 a)."""
    H, a, t0 = 2.0, 1.0, 1.0
    for w in (0.1, 0.5, 1.0, 2.0):
        lam, t = K.window_load_sup([1.0], [t0 - a, t0, t0 + a], [[0.0, H, 0.0]], w, 10.0)
        assert lam == pytest.approx(H * w - H * w * w / (4 * a), rel=1e-12)
        assert t == pytest.approx(t0 - w / 2, abs=1e-9)


def test_constant_rates_reduce():
    """Constant rates: A_j = zeta lam_j min(h / zeta, T - t); the sup is
    zeta lam min(h / zeta, T); p*_k equals the constant-rate continuation
    probabilities."""
    lam = [0.3, 0.2, 0.1]
    f = np.ones((3, 2))
    for zeta, h, T in ((1.0, 5.0, 100.0), (4.0, 8.0, 100.0), (1.0, 50.0, 20.0)):
        Lam, _ = K.window_load_sup(lam, [0.0, 1.0], f, h, T, zeta)
        assert Lam == pytest.approx(zeta * 0.6 * min(h / zeta, T), rel=1e-12)
        A = K.window_arrivals(lam, [0.0, 1.0], f, T - 1.0, h, zeta, T)
        assert A == pytest.approx(zeta * np.array(lam) * min(h / zeta, 1.0), rel=1e-12)
    seg = K.segment_intensities(lam, [0.0, 1.0], f, [8, 20, 40], out_len=[8, 20, 40])
    p = K.continuation_sup(seg, [0.0, 1.0], 100.0)
    ref = K.continuation_probabilities(K.segment_rates(lam, [8, 20, 40], out_len=[8, 20, 40]))
    assert p == pytest.approx(ref, rel=1e-12)


def test_window_sup_brute_force():
    """Random profiles: the exact supremum is at least every grid value of the
    window integral (computed by quadrature) and within the grid's Lipschitz
    slack of the best of them."""
    rng = np.random.default_rng(8)
    for trial in range(6):
        m, T = 2, 100.0
        rt, rf = _rand_profile(rng, m, T, int(rng.integers(2, 9)))
        lam = rng.uniform(0.1, 1.0, m)
        h = float(rng.uniform(1.0, 40.0))
        Lam, _ = K.window_load_sup(lam, rt, rf, h, T)
        tot = lambda u: sum(lam[j] * np.interp(u, rt, rf[j]) for j in range(m))
        grid = np.linspace(0.0, T, 801)
        vals = [integrate.quad(tot, t, min(T, t + h), points=[x for x in rt if t < x < t + h],
                               limit=200)[0] for t in grid]
        lip = 2 * sum(lam) * rf.max()
        assert Lam >= max(vals) - 1e-9
        assert Lam <= max(vals) + lip * (grid[1] - grid[0])


def test_continuation_sup_brute_force():
    """Random profiles: sup of the instantaneous ratio against a dense grid,
    and short windows at the grid's best point approach it."""
    rng = np.random.default_rng(9)
    for trial in range(6):
        T = 50.0
        rt, rf = _rand_profile(rng, 3, T, int(rng.integers(2, 8)))
        rf[:, :] = np.maximum(rf, 0.05)  # keep the denominators positive
        lam = rng.uniform(0.1, 1.0, 3)
        seg = K.profile_intensities(lam, rt, rf)  # one segment per type
        p = K.continuation_sup(seg, rt, T)
        grid = np.linspace(0.0, T, 20001)
        for k in range(2):
            num = seg[k + 1:].sum(axis=0)
            den = seg[k:].sum(axis=0)
            r = np.interp(grid, rt, num) / np.interp(grid, rt, den)
            assert p[k] >= r.max() - 1e-12
            assert p[k] <= r.max() + 1e-3


def test_fluid_throughput_and_batch_time():
    lam, lp = [0.3, 0.1], [8, 20]
    # constant rates: sum lam_j l'_j
    assert K.fluid_throughput_tv(lam, [0.0], [[1.0], [1.0]], lp, 10.0) == pytest.approx(4.4)
    # a profile sampled over whole cycles of 1 + a sin averages to 1 (the
    # trapezoid sum of the sine samples over full periods is zero)
    t = np.linspace(0.0, 30.0, 25)
    f = 1.0 + 0.5 * np.sin(2 * math.pi * 2 * t / 30.0)
    assert K.fluid_throughput_tv(lam, t, [f, f], lp, 30.0) == pytest.approx(4.4, rel=1e-12)
    # hand count: l = 2, segments (1, 3), n = (2, 1): segment 1 holds stages 0
    # and 1 (2 + 3 tokens per prompt), segment 2 stages 2 and 3 (4 + 5)
    assert K.full_batch_time(1.0, 0.5, 2, [1, 3], [2, 1]) == pytest.approx(1.0 + 0.5 * 19)


def test_check_conditions():
    """The cyclic profile at 0.9 of a threshold: the load condition holds;
    doubling the rates breaks it."""
    t = np.linspace(0.0, 1000.0, 25)
    f = np.stack([1.0 + 0.5 * np.sin(2 * math.pi * t / 1000.0 + 2 * math.pi * j / 3)
                  for j in range(3)])
    lam = np.array([0.05, 0.03, 0.02])
    delta = 10.0
    Lam, _ = K.window_load_sup(lam, t, f, delta, 1000.0)
    n1 = Lam / 0.9
    ok = K.check_time_varying(lam, t, f, [n1, 1.0, 1.0], delta, 1000.0)
    assert ok["load_ok"] and ok["Lambda_pi"] == pytest.approx(Lam)
    bad = K.check_time_varying(2 * lam, t, f, [n1, 1.0, 1.0], delta, 1000.0)
    assert not bad["load_ok"]
    seg = K.segment_intensities(lam, t, f, [8, 20, 40], out_len=[8, 20, 40])
    res = K.check_time_varying(lam, t, f, [n1, n1, n1], delta, 1000.0, seg_inten=seg)
    assert len(res["p_star"]) == 2 and res["continuation_ok"]
    res = K.check_time_varying(lam, t, f, [n1, 0.1 * n1, 0.1 * n1], delta, 1000.0,
                               seg_inten=seg)
    assert not res["continuation_ok"]
