"""The paper's throughput statements at scale on the GPU (8192 replicas):

* Theorem 1 on the integer instance (types (2,2), (1,4), rates (3,2),
  d0 0.43, d1 0.01, C = M* = 57, thresholds n* = (3,2), fluid throughput 14):
  with 10 % slack the throughput is the offered load (gap below 0.2 %) and
  nothing is evicted; at the boundary the gap to the fluid throughput shrinks
  as the horizon grows;
* Proposition 3 (one type, l = l' = 1, lam = 4, C = 12, d0 + 12 d1 = 1):
  greedy FCFS stays a constant below the fluid throughput 4 at every horizon,
  while WAIT with n* = 4 closes the gap.
Sampled replicas equal the oracle's."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import sim_module
from tests.parity_util import compare

pytestmark = pytest.mark.gpu

REPS = W.ids(8192)


def _thr(g):
    return float(g["completed_tokens"].sum() / g["t_end"].sum())


def _parity(B, job, g, H, ctx):
    from oracle import oracle as O
    sub = W.Job(job.wl, job.seed, job.replica_ids[[0, 8191]])
    o = O.run_job(sub, H)
    compare({k: v[[0, 8191]] for k, v in g.items()}, o, ctx)


def test_theorem1_integer_instance():
    B = sim_module()
    gaps = {}
    for scale in (0.9, 1.0):
        lam = [3.0 * scale, 2.0 * scale]
        target = 2 * lam[0] + 4 * lam[1]
        wl = W.Workload(prompt_len=[2, 1], lam=lam, d0=0.43, d1=0.01, C=57, policy="wait",
                        n=[3, 2], out_len=[2, 4], hist_edges=W.default_edges(0.43, 64),
                        record_capacity=1 << 18)
        job = W.Job(wl, 0, REPS)
        for H in (10000, 100000):
            print(f"[gpu] theorem 1: scale {scale}, horizon {H}", flush=True)
            g = B.run_batch([job], H)
            assert g["evictions"].sum() == 0 and np.all(g["peak_mem"] <= 57)
            gaps[scale, H] = abs(_thr(g) - target) / target
            if H == 10000:
                _parity(B, job, g, H, f"theorem 1 scale {scale}")
    print(f"[gpu] theorem 1: relative throughput gaps {gaps}", flush=True)
    assert gaps[0.9, 100000] < 0.002
    assert gaps[1.0, 100000] < gaps[1.0, 10000]


def test_proposition3_fcfs_gap():
    B = sim_module()
    d1 = 0.01
    common = dict(prompt_len=[1], lam=[4.0], d0=1.0 - 12 * d1, d1=d1, C=12, out_len=[1],
                  hist_edges=W.default_edges(0.88, 32), record_capacity=1 << 18)
    thr = {}
    for pol, n in (("fcfs", []), ("wait", [4])):
        job = W.Job(W.Workload(policy=pol, n=n, **common), 0, REPS)
        for H in (4000, 64000):
            print(f"[gpu] proposition 3: {pol}, horizon {H}", flush=True)
            g = B.run_batch([job], H)
            thr[pol, H] = _thr(g)
            if pol == "wait":
                assert g["evictions"].sum() == 0
            if H == 4000:
                _parity(B, job, g, H, f"proposition 3 {pol}")
    print(f"[gpu] proposition 3: throughputs {thr}", flush=True)
    assert thr["fcfs", 4000] < 3.7 and thr["fcfs", 64000] < 3.7
    assert thr["wait", 64000] > 3.95
    assert 4.0 - thr["wait", 64000] < 4.0 - thr["wait", 4000]
