"""Side checks of the paper's single-type analysis (Section 4.3):

* the embedded review process of a critical threshold queue: pathwise
  W^B = sum_b X^b - n (B - B_stuck), hence E[W^B] = n E[B_stuck] (the lemma on
  queue length and stuck time), and W^B grows like sqrt(B) (a reflected
  zero-drift walk);
* the square-root law at the boundary (the proposition on the sqrt(T) lower
  bound): WAIT on a single type at critical load (lambda Delta T = n) has mean
  censored latency growing like the square root of the horizon in the oracle,
  while a subcritical load keeps it bounded.
"""
import math

import numpy as np
import pytest

import workloads as W
from paper_2504_11320_amd import analysis as A


def test_review_identity():
    for n in (1, 2, 5):
        r = A.review_process(n, 400, 20000, seed=n)
        B = 400
        assert np.array_equal(r["W"], r["arrivals"] - n * (B - r["stuck"]))
        lhs, rhs = r["W"].mean(), n * r["stuck"].mean()
        se = (r["W"] - n * r["stuck"]).std() / math.sqrt(len(r["W"]))
        assert abs(lhs - rhs) < 5 * se


def test_review_sqrt_growth():
    """E[W^B] for B and 16 B: ratio near 4 (sqrt of 16)."""
    a = A.review_process(2, 250, 20000, seed=1)["W"].mean()
    b = A.review_process(2, 4000, 20000, seed=2)["W"].mean()
    assert 3.4 < b / a < 4.6


def _critical(lam):
    """One type, l = 1, l' = 1, threshold n = 2, d0 = 1, d1 = 0: every batch
    lasts 1, so lam = 2 is the boundary lam Delta T = n."""
    return W.Workload(prompt_len=[1], lam=[lam], d0=1.0, d1=0.0, C=64, policy="wait",
                      n=[2], out_len=[1], hist_edges=W.default_edges(1.0, 8),
                      record_capacity=1 << 14)


def test_sqrt_t_latency_at_the_boundary(oracle_lib):
    from oracle import oracle as O
    reps = W.ids(256)
    lat = {}
    for lam in (2.0, 1.6):
        for H in (500, 8000):
            r = O.run_job(W.Job(_critical(lam), 7, reps), H)
            assert np.all(r["flags"] == 0)
            lat[lam, H] = float((r["lat_area"] / r["arrivals"]).mean())
    crit = lat[2.0, 8000] / lat[2.0, 500]
    sub = lat[1.6, 8000] / lat[1.6, 500]
    assert 2.8 < crit < 5.5, crit      # sqrt(16) = 4
    assert 0.8 < sub < 1.25, sub       # bounded
