"""Pins of the WAIT-no-wait oracle (the threshold-only variant of WAIT in the
paper's appendix on thresholds without waiting): a type is served whenever it
has a waiting or resident prompt, and at most n_j waiting prompts of type j are
admitted per batch."""
import numpy as np

import workloads as W
from tests.parity_util import compare


def _model(policy, n, m=3, C=10**9, lam=(0.02, 0.01, 0.005)):
    return W.Workload(prompt_len=[16, 64, 128][:m], lam=list(lam[:m]), d0=5.0, d1=0.01,
                      C=C, policy=policy, n=list(n), out_len=[8, 20, 40][:m],
                      hist_edges=W.default_edges(5.0, 100), record_capacity=1 << 14)


def test_unlimited_thresholds_equal_fcfs(oracle_lib):
    """With thresholds above any queue length and memory that never binds,
    WAIT-no-wait admits everything waiting and advances every resident at
    every batch, exactly as FCFS does: identical counts, sums equal to
    rounding (the two select the same prompts in a different order)."""
    from oracle import oracle as O
    for m in (1, 3):
        nw = _model("wait-nowait", [1 << 20] * m, m=m)
        fc = _model("fcfs", [], m=m)
        a = O.run_job(W.Job(nw, 3, W.ids(6)), 3000)
        b = O.run_job(W.Job(fc, 3, W.ids(6)), 3000)
        assert np.all(a["evictions"] == 0)
        compare(a, b, f"no-wait vs FCFS, m={m}")


def test_admissions_bounded_by_thresholds(oracle_lib):
    from oracle import oracle as O
    n = [2, 1, 3]
    wl = _model("wait-nowait", n, lam=(0.3, 0.1, 0.05))
    r = O.run_one(wl, 1, 0, 2000, btrace_cap=2000)
    pre = np.array([b["prefills"] for b in r["batches_trace"]])
    assert pre.max() <= sum(n) and pre.max() > 1
    # service never waits: a batch runs whenever anything is waiting or
    # resident, so the only idle waits are on an empty system
    assert r["idle_waits"] <= r["batches"]


def test_hand_trace(oracle_lib):
    """One type, l = 2, l' = 1, n = 2, four requests at t = 0.  Stage times:
    tau = d0 + d1 * tokens.  Batch 1 admits two prompts (tokens 2 + 2 = 4),
    batch 2 decodes them (stage 1, tokens 3 + 3 = 6; they complete) and admits
    the other two (4), batch 3 decodes those (6)."""
    from oracle import oracle as O
    d0, d1 = 1.0, 0.25
    times = [0.0] * 4
    wl = W.trace_workload("wait-nowait", [2], [1], d0, d1, 1000, [2], times, [0] * 4)
    r = O.run_one(wl, 0, 0, 3, btrace_cap=3)
    tok = [b["tokens"] for b in r["batches_trace"]]
    assert tok == [4, 10, 6]
    assert r["completions"] == 4
    tau = [d0 + d1 * x for x in tok]
    # latencies: two complete at the end of batch 2, two at the end of batch 3
    t2, t3 = tau[0] + tau[1], tau[0] + tau[1] + tau[2]
    assert abs(r["lat_completed_sum"] - (2 * t2 + 2 * t3)) < 1e-12
    # WAIT serves a type only when n = 2 prompts wait: after batch 2 nothing
    # waits, the two residents stay frozen and the replica stalls
    wl_w = W.trace_workload("wait", [2], [1], d0, d1, 1000, [2], times, [0] * 4)
    rw = O.run_one(wl_w, 0, 0, 3, btrace_cap=3)
    assert [b["tokens"] for b in rw["batches_trace"]] == [4, 10]
    assert rw["completions"] == 2 and rw["flags"] == 2
    # with 3 requests no-wait serves the third at once and drains everything
    wl3 = W.trace_workload("wait-nowait", [2], [1], d0, d1, 1000, [2], times[:3], [0] * 3)
    a = O.run_one(wl3, 0, 0, 3, btrace_cap=3)
    assert a["completions"] == 3
    assert [x["tokens"] for x in a["batches_trace"]] == [4, 8, 3]
