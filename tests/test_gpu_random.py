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
