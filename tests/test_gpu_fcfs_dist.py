"""FCFS with output lengths drawn per request (Section 4.1's FCFS under the
unknown-length model of Section 5.1) on the GPU, against the oracle.

The kernel keeps residents in admission order with an exit calendar (a
prompt admitted at batch kb with length L completes at kb + L) instead of
the per-type deques of the known-length kernel.  Checked: arrival lists with
tight memory (LIFO evictions, restarts, first-token flags), random models
with drawn lengths and reserves, the Llama-shaped mix with geometric outputs,
per-batch traces batch by batch, a checkpointed resume, and one call mixing
all four launch kinds.
"""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import check, sim_module

pytestmark = pytest.mark.gpu

INT_F = ("tokens", "prefills", "selected", "completions", "evict_pre", "evict_post",
         "mem_after", "waiting_after", "resident_after")


@pytest.fixture(scope="module")
def B():
    return sim_module()


def random_fcfs_dist(rng):
    m = int(rng.integers(1, 5))
    cap = int(rng.integers(2, 40))
    l = [int(x) for x in rng.integers(1, 40, m)]
    cdf = np.stack([W.geometric_cdf_table(float(rng.uniform(1.5, cap)), cap) for _ in range(m)])
    C = int((max(l) + cap) * rng.uniform(1.0, 5.0))
    reserve = float(rng.choice([0.0, 0.01, 0.05]))
    if max(l) > C - int(np.ceil(reserve * C)):
        reserve = 0.0
    return W.Workload(prompt_len=l, lam=[float(x) for x in rng.uniform(0.02, 1.0, m)],
                      d0=float(rng.uniform(0.5, 5.0)), d1=float(rng.uniform(0.0, 0.02)), C=C,
                      policy="fcfs", n=[], out_cap=cap, out_cdf=cdf, reserve=reserve,
                      hist_edges=W.default_edges(1.0, 96), record_capacity=1 << 13)


def test_traces_with_evictions(B):
    rng = np.random.default_rng(5)
    jobs = []
    for x in range(6):
        n = 120
        times = np.sort(rng.uniform(0.0, 60.0, n))
        types = rng.integers(0, 2, n)
        lengths = rng.integers(1, 12, n)
        wl = W.trace_workload("fcfs", [3, 7], None, 1.0, 0.01, 60 + 10 * x, [], times, types,
                              lengths=lengths, out_cap=12, record_capacity=1 << 10)
        jobs.append(W.Job(wl, 0, W.ids(2)))
    g, _ = check(B, jobs, 300, "fcfs drawn lengths, traces")
    assert g["evictions"].sum() > 0


def test_random_models(B):
    rng = np.random.default_rng(17)
    jobs = [W.Job(random_fcfs_dist(rng), 3, W.ids(8)) for _ in range(16)]
    g, _ = check(B, jobs, 2000, "fcfs drawn lengths, random models")
    assert g["evictions"].sum() > 0


def test_llama_mix_geometric_outputs(B):
    jobs = []
    for j in W.config3(replicas=64, rate_index=[8, 31]):
        wl = W.Workload(**{**j.wl.__dict__, "policy": "fcfs", "n": [], "seg_end": None,
                           "reserve": 0.01})
        jobs.append(W.Job(wl, j.seed, j.replica_ids))
    check(B, jobs, 4000, "fcfs drawn lengths, Llama mix")


def test_batch_traces(B):
    from oracle import oracle as O
    rng = np.random.default_rng(23)
    wls = [random_fcfs_dist(rng) for _ in range(4)]
    jobs = [W.Job(wl, 1, W.ids(2)) for wl in wls]
    H = 250
    sim = B.Simulation(jobs)
    sim.prepare()
    tr = sim.advance_traced(H, H)
    res = sim.results()
    r = 0
    for job in jobs:
        for x in range(job.n):
            o = O.run_one(job.wl, job.seed, int(job.replica_ids[x]), H, btrace_cap=H)
            nb = int(res["batches"][r])
            assert nb == o["batches"]
            for b in range(nb):
                for f in INT_F:
                    assert tr[r][b][f] == o["batches_trace"][b][f], (r, b, f)
                for f in ("t_launch", "tau"):
                    y = o["batches_trace"][b][f]
                    assert abs(float(tr[r][b][f]) - y) <= 1e-12 * max(abs(y), 1e-300)
            r += 1


def test_checkpoint_resume(B):
    import torch
    rng = np.random.default_rng(29)
    jobs = [W.Job(random_fcfs_dist(rng), 2, W.ids(6)) for _ in range(5)]
    ref = B.Simulation(jobs)
    ref.run_ex(1500)
    want = ref.results()
    a = B.Simulation(jobs)
    out = torch.empty(32 << 20, dtype=torch.uint8, device="cuda")
    used = a.run_ex(700, state_out=out)
    c = B.Simulation(jobs)
    c.run_ex(800, state_in=out[:used].cpu().to("cuda"))
    got = c.results()
    for k in want:
        assert np.array_equal(want[k], got[k]), k


def test_all_four_launch_kinds_in_one_call(B):
    rng = np.random.default_rng(31)
    jobs = [W.Job(random_fcfs_dist(rng), 4, W.ids(5))]
    jobs += W.config2(replicas=5, rate_index=[20])
    jobs += W.config3(replicas=5, rate_index=[20])
    jobs += [j for j in W.config_pd(replicas=5) if j.wl.policy == "fcfs"][:1]
    check(B, jobs, 1500, "four launch kinds")
