"""The decode-only (prefill-decode disaggregated) workload as a model variant
(the paper's appendix on PD-disaggregated deployment, p630d20): a request
entering with a 630-token context and 20 tokens to generate is the model's
type (l = 630, l' = 19).  Pinned by a single request's latency (the sum of
its 20 decode steps over contexts 630..649) and by the fluid thresholds; the
workload's time constants are chosen here (the appendix's simulator profiles are
not available), so its latency comparison is not asserted."""
import math

import numpy as np
import pytest

import workloads as W


def test_single_request_latency(oracle_lib):
    from oracle import oracle as O
    d0, d1 = 10.0, 5e-5
    # FCFS serves a lone resident at every batch (WAIT would hold it until n
    # more requests wait)
    wl = W.trace_workload("fcfs", [W.PD_CONTEXT], [W.PD_DECODE - 1], d0, d1, 137000, [],
                          [0.0], [0])
    r = O.run_one(wl, 0, 0, 50)
    steps = [d0 + d1 * (W.PD_CONTEXT + i) for i in range(W.PD_DECODE)]
    assert r["completions"] == 1 and r["batches"] == W.PD_DECODE
    assert r["lat_completed_sum"] == pytest.approx(sum(steps), rel=1e-14)
    # generated tokens = model output length + 1
    assert r["completed_tokens"] + r["completions"] == W.PD_DECODE


def test_thresholds_are_the_fluid_ones():
    import oracle.fluid as F
    for lam, n in zip(W.PD_RATES, W.PD_THRESHOLDS):
        st = F.single_type(W.PD_CONTEXT, W.PD_DECODE - 1, lam, 10.0, 5e-5)
        assert st["stable"] and n == math.ceil(st["nstar"])
        # the WAIT condition d0 + d1 M^pi <= n / lam holds and M^pi <= C
        mpi = n * F.stage_work(W.PD_CONTEXT, W.PD_DECODE - 1)
        assert 10.0 + 5e-5 * mpi <= n / lam and mpi <= 137000


def test_both_policies_keep_up(oracle_lib):
    """A small oracle sample at the lowest and highest rates: WAIT never evicts
    (M^pi <= C) and both policies complete requests at the offered rate."""
    from oracle import oracle as O
    jobs = W.config_pd(replicas=8)
    for j in jobs:
        if j.wl.lam[0] not in (W.PD_RATES[0], W.PD_RATES[-1]):
            continue
        r = O.run_job(j, 20000)
        assert np.all(r["flags"] == 0)
        if j.wl.policy == "wait":
            assert np.all(r["evictions"] == 0)
        rate = r["completions"] / r["t_end"]
        assert np.all(np.abs(rate / j.wl.lam[0] - 1.0) < 0.05)
