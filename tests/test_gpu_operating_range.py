"""The stable operating range on the single-type p512d20 workload (the
paper's Section 6 comparison of WAIT with the greedy FCFS baselines, here in
the linear time model with the fluid boundary at 22 requests/s): 7 rates up
to the boundary, 2048 replicas x 5 x 10^4 batches each, WAIT with the fluid
thresholds, FCFS with a 1 % reserve, FCFS with 512-token chunked prefill.

Checked: below the boundary WAIT and FCFS both complete the offered load;
at the boundary WAIT evicts nothing and keeps a lower mean latency than FCFS,
which evicts; the stability point of WAIT (completion rate within 1 % of the
arrival rate) is at least FCFS's.  Sampled replicas equal the oracle's."""
import math

import numpy as np
import pytest

import workloads as W
from paper_2504_11320_amd import analysis as A
from tests.gpu_util import sim_module
from tests.parity_util import compare



def test_thresholds_are_the_fluid_ones():
    import oracle.fluid as F
    for frac, n in zip(W.P512_FRACS, W.P512_THRESHOLDS):
        st = F.single_type(512, 20, frac * W.P512_LAMSTAR, 10.0, W.P512_D1)
        assert st["stable"] and n == math.ceil(st["nstar"] - 1e-9)
    # the boundary: M* = C at 22 requests/s
    st = F.single_type(512, 20, W.P512_LAMSTAR, 10.0, W.P512_D1)
    assert st["Mstar"] == pytest.approx(137000, rel=1e-9)


@pytest.mark.gpu
def test_operating_range():
    B = sim_module()
    from oracle import oracle as O
    H = 50000
    jobs = W.config_p512d20()
    print(f"[gpu] operating range: {len(jobs)} jobs x 2048 replicas x {H}", flush=True)
    g = B.run_batch(jobs, H)
    per = B.split_by_job(g, jobs)
    nr = len(W.P512_FRACS)
    names = ("wait", "fcfs", "fcfs-chunk512")
    rows = {}
    for pi, name in enumerate(names):
        comp, lat, ev = [], [], []
        for ri in range(nr):
            r = per[pi * nr + ri]
            lam = jobs[pi * nr + ri].wl.lam[0]
            comp.append(float(r["completions"].sum() / r["t_end"].sum()))
            lat.append(float(r["lat_completed_sum"].sum() / max(1, r["completions"].sum())))
            ev.append(int(r["evictions"].sum()))
        rows[name] = (comp, lat, ev)
        print(f"[gpu] {name}: completion/arrival "
              f"{[round(c / (f * W.P512_LAMSTAR), 3) for c, f in zip(comp, W.P512_FRACS)]}, "
              f"mean latency {[round(x) for x in lat]}, evictions {ev}", flush=True)
    rates = [f * W.P512_LAMSTAR for f in W.P512_FRACS]
    wc, wl_, we = rows["wait"]
    fc, fl, fe = rows["fcfs"]
    for i in range(nr - 2):   # below the boundary
        assert wc[i] > 0.99 * rates[i] and fc[i] > 0.99 * rates[i]
    assert we[-1] == 0 and fe[-1] > 0
    assert wl_[-1] < fl[-1]
    assert A.lambda_hat(rates, wc, tol=0.01) >= A.lambda_hat(rates, fc, tol=0.01)
    for idx in (nr - 1, 2 * nr - 1, 3 * nr - 1):
        sub = W.Job(jobs[idx].wl, 0, jobs[idx].replica_ids[[0, 2047]])
        o = O.run_job(sub, H)
        start = sum(j.n for j in jobs[:idx])
        compare({k: v[[start, start + 2047]] for k, v in g.items()}, o, f"operating range {idx}")
