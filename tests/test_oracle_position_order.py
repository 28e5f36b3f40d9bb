"""Nested WAIT: the most recently admitted prompt stands first in position
order (Algorithm 2, Section 5.1; Algorithm 4, Appendix B.1).

Cohorts enter a segment from the front of its FIFO boundary queue, every
cohort of a segment leaves it after the same number of services, and the
survivors of one exit join the next queue in admission order; an evicted
prompt re-enters with a new admission key.  So along segment 1, boundary
queue 2, segment 2, ... admission keys only decrease, and the LIFO victim of
either repair lies in the lowest non-empty boundary queue, or, when those
are empty, in the lowest segment that holds a candidate.  The GPU kernel
chooses its victims by that position alone; here the oracle, built with its
position-order counters, confirms at every eviction that its key comparison
lands there (random models with tight memory, per-stage caps, and the
heavy-tailed 10-type and geometric 3-type workloads).
"""
import numpy as np
import pytest

import workloads as W


@pytest.fixture(scope="module")
def checked(tmp_path_factory):
    from oracle import oracle as O
    return O, O.build_order_checked(str(tmp_path_factory.mktemp("ord") / "liboracle_ord.so"))


def _counts(L):
    return [(L.oracle_order_checks(k), L.oracle_order_misses(k)) for k in (0, 1)]


def _run_all(O, L, jobs, horizon, reps):
    before = _counts(L)
    for j in jobs:
        O.run(j.wl, j.seed, j.replica_ids[:reps], horizon, threads=4, library=L)
    after = _counts(L)
    return [(a[0] - b[0], a[1] - b[1]) for a, b in zip(after, before)]


def test_random_models(checked):
    from tests.test_oracle_stage_caps import _random_nested
    O, L = checked
    rng = np.random.default_rng(5)
    jobs = [W.Job(_random_nested(rng), 3, W.ids(4)) for _ in range(16)]
    (bc, bm), (ic, im) = _run_all(O, L, jobs, 1500, 4)
    assert bc > 1000 and ic > 1000, (bc, ic)
    assert bm == 0 and im == 0, (bm, im)


def test_random_models_with_stage_caps(checked):
    from tests.test_gpu_stage_caps import random_capped
    O, L = checked
    rng = np.random.default_rng(6)
    jobs = [W.Job(random_capped(rng), 3, W.ids(4)) for _ in range(16)]
    (bc, bm), (ic, im) = _run_all(O, L, jobs, 1500, 4)
    assert bc > 1000 and ic > 1000, (bc, ic)
    assert bm == 0 and im == 0, (bm, im)


def test_benchmark_workloads(checked):
    O, L = checked
    (bc, bm), (ic, im) = _run_all(O, L, W.config5(replicas=4), 5000, 4)
    assert bc > 100 and ic > 100, (bc, ic)
    assert bm == 0 and im == 0, (bm, im)
    (bc, bm), (ic, im) = _run_all(O, L, W.config3(replicas=4)[::4], 2000, 4)
    assert bc + ic > 100, (bc, ic)
    assert bm == 0 and im == 0, (bm, im)
