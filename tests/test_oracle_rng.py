"""Pins of the oracle's random-number pieces (CPU only).

* Philox4x32-10 against rocRAND's independent implementation of the same
  generator (Salmon et al., SC'11), compiled here as host code.
* ln against the C library logarithm (<= 2 ulp) and exact powers of two.
* Exponential gaps (Poisson arrivals, Section 2.1) by a Kolmogorov-Smirnov
  test; output lengths against their CDF table by a chi-square test.
"""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

from workloads import geometric_cdf_table

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def kat_binary(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available for the rocRAND known-answer helper")
    out = tmp_path_factory.mktemp("kat") / "kat"
    src = os.path.join(HERE, "philox_ref", "rocrand_philox_kat.cpp")
    subprocess.run([hipcc, "-O1", "--offload-host-only", "-o", str(out), src],
                   check=True, capture_output=True)
    return str(out)


def test_philox_matches_rocrand(oracle_lib, kat_binary):
    O = oracle_lib
    rng = np.random.default_rng(12345)
    cases = [[0, 0, 0, 0, 0, 0], [0xFFFFFFFF] * 6, [1, 2, 3, 4, 5, 6]]
    cases += rng.integers(0, 2**32, size=(3000, 6), dtype=np.uint64).tolist()
    # the simulator's counter layout: (k, type, replica, 0), key = seed words
    cases += [[k, j, r, 0, 0, 0] for k in range(5) for j in range(3) for r in (0, 7)]
    inp = "\n".join(" ".join(str(int(x)) for x in c) for c in cases) + "\n"
    res = subprocess.run([kat_binary], input=inp, capture_output=True, text=True,
                         check=True)
    ref = [list(map(int, line.split())) for line in res.stdout.strip().splitlines()]
    assert len(ref) == len(cases)
    for c, r in zip(cases, ref):
        got = O.philox(c[:4], c[4:]).tolist()
        assert got == r, (c, got, r)


def test_uniform_extremes(oracle_lib):
    O = oracle_lib
    assert O.uniform(0, 0) == 2.0 ** -53
    assert O.uniform(0xFFFFFFFF, 0xFFFFFFFF) == 1.0 - 2.0 ** -53
    # the low 12 bits of w1 are not used; bit 12 of w1 is the lowest used bit
    assert O.uniform(0, 0xFFF) == 2.0 ** -53
    assert O.uniform(0, 0x1000) == 3.0 * 2.0 ** -53
    assert O.uniform(0x80000000, 0) == 0.5 + 2.0 ** -53


def _ulps(a, b):
    return abs(a - b) / math.ulp(b)


def test_ln_within_two_ulp(oracle_lib):
    O = oracle_lib
    rng = np.random.default_rng(7)
    us = list(rng.random(100000))
    us += [2.0 ** -53, 1.0 - 2.0 ** -53, 0.5, math.sqrt(0.5), math.sqrt(0.5) * (1 + 2e-16),
           math.sqrt(0.5) * (1 - 2e-16), 0.75, 0.999999, 1e-10, 1e-16]
    us += list(10.0 ** rng.uniform(-15.9, 0, 20000))
    worst = 0.0
    for u in us:
        if not (0.0 < u < 1.0):
            continue
        worst = max(worst, _ulps(O.ln(u), math.log(u)))
    assert worst <= 2.0, worst


def test_ln_powers_of_two(oracle_lib):
    O = oracle_lib
    for k in range(1, 54):
        assert _ulps(O.ln(2.0 ** -k), -k * math.log(2.0)) <= 1.0


def test_gaps_are_exponential(oracle_lib):
    O = oracle_lib
    lam = 0.37
    gaps = np.array([O.draw(0, 3, 1, k, lam)[0] for k in range(20000)])
    assert np.all(gaps > 0)
    ks = stats.kstest(gaps, "expon", args=(0, 1.0 / lam))
    assert ks.pvalue > 1e-3, ks
    # independent streams across types and replicas
    other = np.array([O.draw(0, 4, 1, k, lam)[0] for k in range(20000)])
    assert abs(np.corrcoef(gaps, other)[0, 1]) < 0.03
    other = np.array([O.draw(0, 3, 2, k, lam)[0] for k in range(20000)])
    assert abs(np.corrcoef(gaps, other)[0, 1]) < 0.03


def test_gaps_scale_with_rate(oracle_lib):
    """Common random numbers across rates: the uniform is the same and the gap
    scales as 1/lambda (division is correctly rounded)."""
    O = oracle_lib
    for k in range(50):
        g1 = O.draw(5, 1, 0, k, 1.0)[0]
        g2 = O.draw(5, 1, 0, k, 0.25)[0]
        assert g2 == g1 / 0.25


def test_output_length_table(oracle_lib):
    O = oracle_lib
    cap = 2048
    row = geometric_cdf_table(64.0, cap)
    Ls = np.array([O.draw(0, 9, 0, k, 1.0, row, cap)[1] for k in range(40000)])
    assert Ls.min() >= 1 and Ls.max() <= cap
    # pmf implied by the table
    T = np.concatenate([[0], row.astype(np.float64), [2.0 ** 32]]) / 2.0 ** 32
    pmf = np.diff(T)[: cap]                       # P(L = s), s = 1..cap
    edges = [1, 8, 16, 32, 48, 64, 96, 128, 192, 256, cap + 1]
    obs = np.array([((Ls >= a) & (Ls < b)).sum() for a, b in zip(edges[:-1], edges[1:])])
    exp = np.array([pmf[a - 1:b - 1].sum() for a, b in zip(edges[:-1], edges[1:])]) * len(Ls)
    chi = ((obs - exp) ** 2 / exp).sum()
    assert stats.chi2.sf(chi, len(obs) - 1) > 1e-3, (obs, exp)
    assert abs(Ls.mean() - 64.0) < 2.0
