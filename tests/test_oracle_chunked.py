"""Pins of the oracle's FCFS with chunked prefill (the Sarathi-style baseline
of Section 6: at most `chunk` prefill tokens per iteration, partial prefills
interleaved with decode work).

* a budget no batch can exhaust reproduces plain FCFS bit for bit;
* hand traces: one long prompt split over two iterations; two prompts sharing
  one budget; a partially prefilled prompt evicted first by the LIFO repair;
* invariants on random models: per-iteration prefill tokens never exceed the
  budget, and the iteration time stays below the no-chunking bound.
"""
import numpy as np
import pytest

import workloads as W
from tests.parity_util import compare


def _trace(l, lp, C, chunk, times, types, d0=1.0, d1=0.01):
    wl = W.trace_workload("fcfs", l, lp, d0, d1, C, [], times, types)
    wl.chunk = chunk
    return wl


def test_unbounded_budget_is_plain_fcfs(oracle_lib):
    from oracle import oracle as O
    from tests.test_gpu_random import random_workload
    rng = np.random.default_rng(5)
    n = 0
    while n < 8:
        wl = random_workload(rng)
        if wl.policy != "fcfs":
            continue
        n += 1
        a = O.run_job(W.Job(wl, 3, W.ids(5)), 1500)
        wl.chunk = 1 << 30
        b = O.run_job(W.Job(wl, 3, W.ids(5)), 1500)
        for f in O.INT_FIELDS + O.F64_FIELDS:
            assert np.array_equal(a[f], b[f]), f
        assert np.array_equal(a["hist"], b["hist"])


def test_one_long_prompt(oracle_lib):
    """l = 1000, l' = 2, chunk 512: iteration tokens 512 (first chunk), 1000
    (the cache after the second), then stages 1 and 2 (1001, 1002)."""
    from oracle import oracle as O
    wl = _trace([1000], [2], 5000, 512, [0.0], [0])
    r = O.run_one(wl, 0, 0, 10, btrace_cap=10)
    tok = [b["tokens"] for b in r["batches_trace"]]
    assert tok == [512, 1000, 1001, 1002]
    assert r["completions"] == 1 and r["batches"] == 4
    assert r["lat_completed_sum"] == pytest.approx(sum(1.0 + 0.01 * x for x in tok), rel=1e-14)
    mem = [b["mem_after"] for b in r["batches_trace"]]
    assert mem == [512, 1001, 1002, 0]


def test_two_prompts_share_the_budget(oracle_lib):
    """Two prompts of 300 at t = 0, l' = 1, chunk 512: A whole (300) and B's
    first 212 tokens; then A's stage 1 (301) and B's last 88 (cache 300);
    then B's stage 1."""
    from oracle import oracle as O
    wl = _trace([300], [1], 5000, 512, [0.0, 0.0], [0, 0])
    r = O.run_one(wl, 0, 0, 10, btrace_cap=10)
    bt = r["batches_trace"]
    assert [b["tokens"] for b in bt] == [300 + 212, 301 + 300, 301]
    assert [b["prefills"] for b in bt] == [2, 1, 0]
    assert [b["completions"] for b in bt] == [0, 1, 1]
    tau = [1.0 + 0.01 * b["tokens"] for b in bt]
    assert r["lat_completed_sum"] == pytest.approx((tau[0] + tau[1]) + sum(tau), rel=1e-14)


def test_partial_prompt_evicted_first(oracle_lib):
    """40 one-token prompts decoding (l' = 100) and a 300-token prompt
    admitted in iteration 2 with chunk 50, C = 400: after iteration 5 the 40
    decoders hold 240 and the partial prompt 200 (440 > 400); LIFO evicts the
    partial prompt (no decode tokens lost) and memory falls to 240."""
    from oracle import oracle as O
    wl = _trace([1, 300], [100, 1], 400, 50, [0.0] * 40 + [1e-9], [0] * 40 + [1])
    r = O.run_one(wl, 0, 0, 5, btrace_cap=5)
    bt = r["batches_trace"]
    assert [b["prefills"] for b in bt] == [40, 1, 1, 1, 1]
    assert [b["mem_after"] for b in bt] == [80, 170, 260, 350, 240]
    assert bt[4]["evict_post"] == 1 and r["evictions"] == 1 and r["evicted_tokens"] == 0
    assert r["waiting_end"] == 1 and r["resident_end"] == 40


def test_budget_and_time_bounds(oracle_lib):
    """Random FCFS models with chunk 16: an iteration processes the resident
    memory (at most C after the repair) plus at most 16 new prefill tokens,
    so its token count never exceeds C + 16."""
    from oracle import oracle as O
    from tests.test_gpu_random import random_workload
    rng = np.random.default_rng(9)
    n = 0
    while n < 6:
        wl = random_workload(rng)
        if wl.policy != "fcfs":
            continue
        n += 1
        wl.chunk = 16
        r = O.run_one(wl, 1, 0, 800, btrace_cap=800)
        for b in r["batches_trace"]:
            assert b["tokens"] <= wl.C + 16
        assert r["completions"] > 0
