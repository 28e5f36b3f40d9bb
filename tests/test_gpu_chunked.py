"""GPU parity of FCFS with chunked prefill (the Sarathi-style baseline of
Section 6) against the oracle: random models at several budgets, the hand
traces of the oracle's pins, an unexhaustible budget equal to plain FCFS, and
resume."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import check, sim_module

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    return sim_module()


def _fcfs_models(seed, count):
    from tests.test_gpu_random import random_workload
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        wl = random_workload(rng)
        if wl.policy == "fcfs":
            out.append(wl)
    return out, rng


def test_random_budgets(B):
    models, rng = _fcfs_models(41, 18)
    jobs = []
    for i, wl in enumerate(models):
        wl.chunk = [1, 7, 16, 64, 512, 3][i % 6]
        jobs.append(W.Job(wl, int(rng.integers(0, 2**63)), W.ids(int(rng.integers(1, 60)))))
    check(B, jobs, 900, "FCFS chunked prefill, 18 random models")


def test_llama_mix_chunk_512(B):
    """The Llama-shaped 3-type mix (prompts 128/512/1024) under FCFS with a
    1 % reserve and 512-token chunks, at three rates."""
    jobs = []
    for ri in (0, 16, 31):
        wl = W.config2(replicas=1, rate_index=[ri])[0].wl
        wl.policy, wl.n, wl.reserve, wl.chunk = "fcfs", [], 0.01, 512
        jobs.append(W.Job(wl, 0, W.ids(45)))
    check(B, jobs, 3000, "FCFS chunk 512, Llama mix, 3 rates x45 x3000")


def test_hand_traces(B):
    tr = []
    a = W.trace_workload("fcfs", [1000], [2], 1.0, 0.01, 5000, [], [0.0], [0])
    a.chunk = 512
    b = W.trace_workload("fcfs", [300], [1], 1.0, 0.01, 5000, [], [0.0, 0.0], [0, 0])
    b.chunk = 512
    c = W.trace_workload("fcfs", [1, 300], [100, 1], 1.0, 0.01, 400, [],
                         [0.0] * 40 + [1e-9], [0] * 40 + [1])
    c.chunk = 50
    g, o = check(B, [W.Job(a, 0, W.ids(1)), W.Job(b, 0, W.ids(1)), W.Job(c, 0, W.ids(1))],
                 5, "chunked prefill hand traces")
    assert g["evictions"][2] == 1 and g["resident_end"][2] == 40


def test_unexhaustible_budget_is_fcfs(B):
    models, _ = _fcfs_models(43, 6)
    jobs0 = [W.Job(wl, 5, W.ids(20)) for wl in models]
    g0 = B.run_batch(jobs0, 1000)
    import dataclasses
    jobs1 = [W.Job(dataclasses.replace(wl, chunk=1 << 30), 5, W.ids(20)) for wl in models]
    g1 = B.run_batch(jobs1, 1000)
    for k in g0:
        assert np.array_equal(g0[k], g1[k]), k


def test_resume(B):
    models, _ = _fcfs_models(47, 4)
    for wl in models:
        wl.chunk = 8
    jobs = [W.Job(wl, 9, W.ids(17)) for wl in models]
    one = B.run_batch(jobs, 800)
    sim = B.Simulation(jobs)
    sim.prepare()
    sim.advance(400, resume=False)
    sim.advance(400, resume=True)
    two = sim.results()
    for k in one:
        assert np.array_equal(one[k], two[k]), k
