"""Pins of the segment-design memory bound in the host calculator (the
decomposition M_req = M^pi + deterministic boundary term + logarithmic buffer
of the segment-wise design, the theta_k roots, fluid thresholds meeting the
segment conditions, and the decomposition against the number of segments)."""
import math

import numpy as np
import pytest

from paper_2504_11320_amd import calibrate as K


def test_agrees_with_the_oracle_formulas():
    """Against the oracle's independent implementation (bisection for theta)
    on random inputs."""
    import oracle.fluid as F
    rng = np.random.default_rng(3)
    for _ in range(25):
        L = int(rng.integers(1, 6))
        seg_end = sorted(rng.choice(np.arange(1, 400), L, replace=False).tolist())
        p = rng.uniform(0.05, 0.9, L - 1).tolist()
        n = [float(rng.uniform(1, 8))]
        for x in p:
            n.append(n[-1] * min(x + float(rng.uniform(0.01, 0.2)), 0.99))
        l = float(rng.uniform(10, 800))
        a = K.memory_requirement(n, seg_end, l, p, 10, float(rng.uniform(1e2, 1e7)), 5.0,
                                 float(rng.uniform(1e-6, 0.1)))
        zT = 1e5
        b = F.nested_m_req(n, seg_end, l, p, 10, zT, 5.0, 1e-3)
        a2 = K.memory_requirement(n, seg_end, l, p, 10, zT, 5.0, 1e-3)
        assert a2["total"] == pytest.approx(b["Mreq"], rel=1e-12)
        assert a2["term1"] == pytest.approx(b["Mpi"], rel=1e-14)
        assert np.allclose(a2["theta"], b["theta"], rtol=1e-10)
        assert a["term1"] == a2["term1"]


def test_theta_root_equation_and_bound():
    """exp(-theta n_k)(1 - p + p e^theta)^{n_{k-1}} = 1 at the root, and
    theta_k >= 8 (n_k - n_{k-1} p_k) / n_{k-1} (the lower bound the theorem
    states)."""
    for nk, nprev, p in ((2.0, 4.0, 0.4), (1.0, 2.0, 0.45), (3.0, 3.5, 0.8),
                         (0.5, 10.0, 0.01), (7.0, 8.0, 0.5)):
        th = K.theta_root(nk, nprev, p)
        val = -th * nk + nprev * math.log(1 - p + p * math.exp(th))
        assert abs(val) < 1e-12 * max(1.0, th * nk)
        assert th >= 8 * (nk - nprev * p) / nprev * (1 - 1e-12)
    with pytest.raises(ValueError):
        K.theta_root(1.0, 2.0, 0.6)   # n_{k-1} p >= n_k: no positive root


def test_one_segment_is_single_type_wait():
    """L = 1: M^pi = n (l'+1)(l + l'/2), the single-type WAIT memory, and no
    boundary terms."""
    r = K.memory_requirement([3.0], [20], 512, [], 1, 1e5, 5.0, 1e-3)
    assert r["term1"] == pytest.approx(3.0 * K.stage_work(512, 20))
    assert r["term2"] == 0.0 and r["term3"] == 0.0


def test_fluid_thresholds_meet_the_conditions():
    rates = [0.02, 0.01, 0.006, 0.004]
    seg_end = [16, 64, 256, 1024]
    n = K.fluid_segment_thresholds(rates, seg_end, 128, 15.0, 0.0001)
    p = K.continuation_probabilities(rates)
    assert 15.0 + 0.0001 * K.base_memory(n, seg_end, 128) < n[0] / sum(rates)
    for k in range(1, 4):
        assert p[k - 1] < n[k] / n[k - 1] < 1
    assert K.fluid_segment_thresholds(rates, seg_end, 128, 15.0, 1.0) is None


def test_decomposition_against_segments():
    """A long-tailed output law (geometric, mean 80, 500 classes): the base
    term falls from L = 1 as segments stop charging short requests for long
    ones, the boundary terms grow with L, and the total is U-shaped (its
    minimum strictly inside the range)."""
    lens = np.arange(1, 501)
    w = np.exp(-lens / 80.0)
    rates = list(0.05 * w / w.sum())
    rows = K.memory_vs_segments(128, list(lens), rates, [1, 2, 3, 4, 6, 8, 12, 16, 24, 32],
                                5.0, 0.00005, 1e5, 1e-3)
    Ls = [r["L"] for r in rows]
    assert Ls[0] == 1 and Ls[-1] >= 24
    t1 = [r["term1"] for r in rows]
    t23 = [r["term2"] + r["term3"] for r in rows]
    tot = [r["total"] for r in rows]
    assert t1[0] > 2 * min(t1)
    assert t23[0] == 0.0 and all(b >= a for a, b in zip(t23[1:], t23[2:]))
    i = int(np.argmin(tot))
    assert 0 < i < len(tot) - 1
    for r in rows:
        assert r["seg_end"] == sorted(set(r["seg_end"])) and r["seg_end"][-1] == 500


def test_equal_rate_cuts():
    cuts = K.equal_rate_cuts([5, 10, 20, 40], [0.25, 0.25, 0.25, 0.25], 4)
    assert cuts == [5, 10, 20, 40]
    assert K.equal_rate_cuts([5, 10, 20, 40], [0.7, 0.1, 0.1, 0.1], 2) == [5, 40]
    assert K.equal_rate_cuts([5, 10, 20, 40], [1, 1, 1, 1], 1) == [40]
