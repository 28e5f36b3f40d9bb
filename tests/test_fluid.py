"""Pins of the fluid/threshold calculator against numbers the paper prints."""
import json
import math
import os

import numpy as np
import pytest

from oracle import fluid as F
import workloads as W

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_lmsys_table_follows_fluid_formula():
    """Section 6.2 table: M*(lam) = d0 A/(1-d1 A) with A = lam E[S], i.e.
    x lam / (1 - y lam).  Fit (x, y) on two rows, predict the other two and
    the crossing with C."""
    g = _gold("lmsys_mstar_table.json")
    (l1, m1), (l2, m2), (l3, m3), (l4, m4) = g["rows"]
    # m = x l / (1 - y l)  ->  x l - m y l = m : linear in (x, y)
    A = np.array([[l1, m1 * l1], [l2, m2 * l2]], dtype=float)
    x, y = np.linalg.solve(A, [m1, m2])
    ES = 1000.0                                   # any E[S]; d0, d1 follow
    d0, d1 = x / ES, y / ES
    for lam, m in ((l3, m3), (l4, m4)):
        pred = F.fluid_mean_work(ES, lam, d0, d1)
        assert abs(pred - m) / m < 5e-4
    cross = g["C"] / ((d0 + d1 * g["C"]) * ES)
    assert cross == pytest.approx(F.lambda_star(ES, d0, d1, g["C"]))
    assert abs(cross - g["crossing"]) < 0.1


@pytest.mark.parametrize("d1", [0.001, 0.01, 0.03, 1.0 / 25])
def test_fcfs_instance_fluid(d1):
    g = _gold("wait_fluid_composition.json")
    d0 = 1.0 - 12.0 * d1
    s = F.single_type(1, 1, 4.0, d0, d1)
    assert s["nstar"] == pytest.approx(g["nstar"], rel=1e-12)
    assert s["Mstar"] == pytest.approx(g["Mstar"], rel=1e-12)
    assert s["throughput"] == 4.0
    m = F.fluid([1], [1], [4.0], d0, d1)
    assert m["Mstar"] == pytest.approx(s["Mstar"], rel=1e-12)
    assert m["dTstar"] == pytest.approx(g["tau"], rel=1e-12)


def test_prop1_instability_threshold():
    # lam d1 (l'+1)(l+l'/2) >= 1 gives no finite equilibrium
    l, lp, d1 = 32, 16, 0.01
    lam_crit = 1.0 / (d1 * F.stage_work(l, lp))
    assert F.single_type(l, lp, lam_crit * 0.999, 5.0, d1)["stable"]
    assert not F.single_type(l, lp, lam_crit * 1.001, 5.0, d1)["stable"]
    # configuration 1: d1 A = 2.08
    wl = W.config1()[0].wl
    A = F.load_A(wl.prompt_len, wl.out_len, wl.lam)
    assert wl.d1 * A == pytest.approx(2.08)


def test_integer_fluid_instance():
    """Types (2,2),(1,4), lam (3,2), d0 0.43, d1 0.01: A = 57, dT* = 1,
    n* = (3, 2), M* = 57 (closed forms of Section 3.2)."""
    f = F.fluid([2, 1], [2, 4], [3.0, 2.0], 0.43, 0.01)
    assert f["A"] == pytest.approx(57.0)
    assert f["dTstar"] == pytest.approx(1.0)
    assert f["nstar"] == pytest.approx([3.0, 2.0])
    assert f["Mstar"] == pytest.approx(57.0)
    assert f["throughput"] == pytest.approx(14.0)
    c = F.wait_conditions([3, 2], [2, 1], [2, 4], [3.0, 2.0], 0.43, 0.01, 57)
    assert c["Mpi"] == pytest.approx(57.0) and c["holds"]


def test_calibration_example():
    g = _gold("calibration_two_segment.json")
    r = F.calibrate(g["tl"], g["widths"], g["p"], g["eta"])
    assert r["n"][1] / r["n"][0] == pytest.approx(0.3)
    assert sum(r["B"]) == pytest.approx(g["tl"])
    assert [round(b) for b in r["B"]] == g["caps_rounded"]
    assert r["B"] == pytest.approx([20.6897, 9.3103], abs=1e-4)


@pytest.mark.parametrize("nk,nkm1,p", [(1, 2, 0.3), (1, 2, 0.01), (2, 4, 0.2),
                                       (3, 4, 0.5), (5, 10, 0.1)])
def test_theta_root(nk, nkm1, p):
    th = F.theta_root(nk, nkm1, p)
    assert math.exp(-th * nk) * (1 - p + p * math.exp(th)) ** nkm1 == pytest.approx(1.0, rel=1e-9)
    assert th >= 8.0 * (nk - nkm1 * p) / nkm1 * (1 - 1e-9)


def test_segment_delta_sbar_and_mpi():
    # one segment covering 0..l' reproduces the WAIT stage work
    assert F.nested_mpi([3], [10], 7) == pytest.approx(3 * F.stage_work(7, 10))
    # two segments r = (1, 2): delta = (2, 1), sbar = (0.5, 2)
    assert F.seg_delta_sbar([1, 2]) == [(2, 0.5), (1, 2.0)]
    assert F.nested_mpi([4, 2], [1, 2], 1) == pytest.approx(18.0)


def test_workload_rate_literals():
    """The rate scales stored with the workloads are the fluid boundary of
    their mixes: M*(Lam*) = C."""
    es2 = sum(p * F.stage_work(l, lp) for p, l, lp in zip(W.C2_MIX, W.C2_PROMPTS, W.C2_OUTPUTS))
    assert W.LAM_STAR_C2 == pytest.approx(F.lambda_star(es2, 15.0, 0.05, 131072), rel=1e-12)
    assert F.fluid_mean_work(es2, W.LAM_STAR_C2, 15.0, 0.05) == pytest.approx(131072, rel=1e-9)

    def es_from_tables(prompts, mix, cdf, cap):
        total = 0.0
        s = np.arange(1, cap + 1, dtype=np.float64)
        for l, p, row in zip(prompts, mix, cdf):
            T = np.concatenate([[0.0], row.astype(np.float64), [2.0 ** 32]]) / 2.0 ** 32
            pmf = np.diff(T)
            total += p * float(np.sum(pmf * (s + 1.0) * (l + s / 2.0)))
        return total

    j3 = W.config3(replicas=1, n_rates=32, rate_index=[0])[0].wl
    es3 = es_from_tables(j3.prompt_len, W.C2_MIX, j3.out_cdf, j3.out_cap)
    assert W.LAM_STAR_C3 == pytest.approx(F.lambda_star(es3, 15.0, 0.05, 131072), rel=1e-6)
    j5 = W.config5(replicas=1)[0].wl
    es5 = es_from_tables(j5.prompt_len, [0.1] * 10, j5.out_cdf, j5.out_cap)
    assert W.LAM_STAR_C5 == pytest.approx(F.lambda_star(es5, 15.0, 0.05, 262144), rel=1e-6)
    assert j5.prompt_len == [108, 176, 235, 296, 365, 446, 549, 692, 924, 1504]


def test_nested_memory_requirement_terms():
    r = F.nested_m_req([4, 2], [4, 8], 4, [0.3], m=2, zeta_T=1e4, d0=1.0, delta=0.1)
    assert r["Mpi"] == pytest.approx(204.0)
    assert r["term2"] == pytest.approx(16.0)
    assert r["term3"] > 0 and r["Mreq"] == pytest.approx(r["Mpi"] + r["term2"] + r["term3"])
