"""GPU parity on seeded random small models across all three policies."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import check, sim_module

pytestmark = pytest.mark.gpu


def random_workload(rng):
    policy = ["wait", "fcfs", "nested", "wait-nowait"][rng.integers(4)]
    m = int(rng.integers(1, 4))
    l = [int(x) for x in rng.integers(1, 40, m)]
    lam = [float(x) for x in rng.uniform(0.02, 1.0, m)]
    d0 = float(rng.uniform(0.5, 5.0))
    d1 = float(rng.uniform(0.0, 0.02))
    edges = W.default_edges(d0, int(rng.integers(1, 120)))
    if policy == "nested":
        cap = int(rng.integers(2, 30))
        nseg = int(rng.integers(1, min(4, cap) + 1))
        cuts = sorted(rng.choice(np.arange(1, cap), size=nseg - 1, replace=False).tolist())
        seg_end = [int(c) for c in cuts] + [cap]
        n = [int(x) for x in rng.integers(1, 4, nseg)]
        cdf = np.stack([W.geometric_cdf_table(float(rng.uniform(1.5, cap)), cap)
                        for _ in range(m)])
        C = int((max(l) + cap) * rng.uniform(1.0, 6.0))
        return W.Workload(prompt_len=l, lam=lam, d0=d0, d1=d1, C=C, policy=policy, n=n,
                          out_cap=cap, out_cdf=cdf, seg_end=seg_end, hist_edges=edges,
                          record_capacity=1 << 14)
    lp = [int(x) for x in rng.integers(1, 25, m)]
    n = [int(x) for x in rng.integers(1, 5, m)] if policy.startswith("wait") else []
    C = int(max(a + b for a, b in zip(l, lp)) * rng.uniform(1.0, 6.0))
    reserve = float(rng.choice([0.0, 0.01, 0.05])) if policy == "fcfs" else 0.0
    if policy == "fcfs" and max(l) > C - int(np.ceil(reserve * C)):
        reserve = 0.0
    return W.Workload(prompt_len=l, lam=lam, d0=d0, d1=d1, C=C, policy=policy, n=n,
                      out_len=lp, reserve=reserve, hist_edges=edges,
                      record_capacity=1 << 14)


def test_random_models():
    B = sim_module()
    rng = np.random.default_rng(2026)
    jobs = []
    for i in range(36):
        wl = random_workload(rng)
        jobs.append(W.Job(wl, int(rng.integers(0, 2**63)), W.ids(int(rng.integers(1, 70)))))
    check(B, jobs, 700, "36 random models, one launch per policy")


def test_wait_nowait_sweep():
    """WAIT-no-wait on the Llama-shaped 3-type mix (thresholds 2, 1, 1) at
    three rates, ragged replica counts, against the oracle."""
    B = sim_module()
    jobs = []
    for ri in (0, 16, 31):
        wl = W.config2(replicas=1, rate_index=[ri])[0].wl
        wl.policy = "wait-nowait"
        wl.n = [2, 1, 1]
        jobs.append(W.Job(wl, 0, W.ids(70)))
    check(B, jobs, 3000, "WAIT-no-wait, 3 rates x70 x3000")


@pytest.mark.parametrize("m", [1, 2, 3, 4, 6, 8])
def test_unit_thresholds(m):
    """WAIT and WAIT-no-wait launches whose jobs all have n_j = 1 run the
    unit-threshold kernels (at most one admission and one completion per type
    and batch): random models with m types against the oracle, at 8 replicas
    per wavefront; a launch of 66,000 replicas (64 per wavefront with 6 or 8
    types, 32 with fewer) gives the same replicas bit-identical results."""
    B = sim_module()
    rng = np.random.default_rng(500 + m)
    jobs = []
    for i in range(6):
        l = [int(x) for x in rng.integers(1, 60, m)]
        lp = [int(x) for x in rng.integers(1, 30, m)]
        wl = W.Workload(prompt_len=l, lam=[float(x) for x in rng.uniform(0.02, 0.6, m)],
                        d0=float(rng.uniform(0.5, 5.0)), d1=float(rng.uniform(0.0, 0.02)),
                        C=int(max(a + b for a, b in zip(l, lp)) * rng.uniform(1.0, 4.0)),
                        policy="wait" if i % 3 else "wait-nowait", n=[1] * m, out_len=lp,
                        hist_edges=W.default_edges(1.0, int(rng.integers(1, 100))),
                        record_capacity=1 << 14)
        jobs.append(W.Job(wl, int(rng.integers(0, 2**63)), W.ids(int(rng.integers(1, 40)))))
    check(B, jobs, 1500, f"unit thresholds, {m} types")
    R = 11000
    g = B.run_batch([W.Job(j.wl, j.seed, W.ids(R)) for j in jobs], 600)
    picks = np.concatenate([np.arange(5), np.arange(R - 5, R)]).astype(np.uint32)
    small = B.run_batch([W.Job(j.wl, j.seed, picks) for j in jobs], 600)
    idx = np.concatenate([R * k + picks.astype(np.int64) for k in range(len(jobs))])
    for k in g:
        assert np.array_equal(g[k][idx], small[k]), k


def test_large_cohorts_under_tight_memory():
    """WAIT and WAIT-no-wait with thresholds up to 16 and memory just above
    the largest request: a service admits a whole cohort and the repair
    evicts most of it again, several prompts of one cohort at a time; every
    field against the oracle."""
    B = sim_module()
    rng = np.random.default_rng(4242)
    jobs = []
    for i in range(16):
        m = int(rng.integers(1, 4))
        l = [int(x) for x in rng.integers(1, 60, m)]
        lp = [int(x) for x in rng.integers(1, 30, m)]
        n = [int(x) for x in rng.integers(2, 17, m)]
        C = int(max(a + b for a, b in zip(l, lp)) * rng.uniform(1.0, 2.5))
        wl = W.Workload(prompt_len=l, lam=[float(x) for x in rng.uniform(0.1, 1.0, m)],
                        d0=float(rng.uniform(0.5, 3.0)), d1=float(rng.uniform(0.0, 0.02)),
                        C=C, policy="wait" if i % 4 else "wait-nowait", n=n, out_len=lp,
                        hist_edges=W.default_edges(1.0, 64), record_capacity=1 << 16)
        jobs.append(W.Job(wl, int(rng.integers(0, 2**63)), W.ids(int(rng.integers(8, 40)))))
    g, _ = check(B, jobs, 1500, "WAIT, cohorts up to 16, tight memory")
    assert g["evictions"].sum() > g["batches"].sum()  # more than one eviction per batch
    assert (g["flags"] == 0).all()
