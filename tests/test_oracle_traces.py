"""Hand traces: the oracle reproduces the batch sequences the paper derives.

Arrivals are injected (trace mode) so every batch is fixed by the paper's
arithmetic: Example 1, the FCFS warm-up and cycle of the proof of
Proposition 3, the WAIT fluid composition of Example 2, and a two-segment
Nested WAIT instance whose full prefix batch equals M^pi.
"""
import json
import os

import pytest

from oracle import fluid as F
from workloads import trace_workload

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_fcfs_cycle_of_proposition_3(oracle_lib):
    O = oracle_lib
    g = _gold("fcfs_cycle_prop3.json")
    d1 = g["instance"]["d1"]
    d0 = 1.0 - 12.0 * d1
    extra = 40                         # "L" of the proof: queue never drains
    times = [1e-4 * i for i in range(extra + 12)]
    wl = trace_workload("fcfs", [1], [1], d0, d1, 12, [], times, [0] * len(times),
                        record_capacity=4096)
    nb = len(g["batches"])
    r = O.run_one(wl, 0, 0, nb, btrace_cap=nb)
    bt = r["batches_trace"]
    for want, got in zip(g["batches"], bt):
        assert got["prefills"] == want["prefills"]
        assert got["selected"] - got["prefills"] == want["decodes"]
        assert got["evict_post"] == want["evicted_after"]
        assert got["completions"] == want["completions"]
        assert got["evict_pre"] == 0
    for got in bt[1:]:
        assert got["tau"] == pytest.approx(1.0, abs=1e-12)
        assert got["tokens"] == 12
    # the cycle completes 6 prompts every 2 time units
    cyc = bt[3:7]
    assert sum(b["completions"] for b in cyc) / sum(b["tau"] for b in cyc) == g["cycle_throughput"]


def test_wait_fluid_composition(oracle_lib):
    O = oracle_lib
    g = _gold("wait_fluid_composition.json")
    d1 = g["instance"]["d1"]
    d0 = 1.0 - 12.0 * d1
    times = [1e-4 * i for i in range(80)]
    wl = trace_workload("wait", [1], [1], d0, d1, 12, [g["nstar"]], times, [0] * 80)
    r = O.run_one(wl, 0, 0, 10, btrace_cap=10)
    bt = r["batches_trace"]
    assert bt[0]["prefills"] == 4 and bt[0]["selected"] == 4
    for b in bt[1:]:
        assert b["prefills"] == 4 and b["selected"] == 8
        assert b["tokens"] == g["batch_tokens"]
        assert b["tau"] == pytest.approx(g["tau"], abs=1e-12)
        assert b["completions"] == g["completions_per_batch"]
        assert b["evict_post"] == 0
    # launch memory of the full batch: 4 prefills (1 each) + 4 decodes (2 each)
    assert r["peak_mem"] == g["Mstar"]
    assert r["evictions"] == 0


def test_example_1_memory_growth(oracle_lib):
    """Example 1: three prompts decoding (3 x 2 = 6 units) and six admitted
    prefills (6 x 1) fill C = 12; afterwards the three complete and the six
    newly prefilled prompts need 6 x 2 = 12 units."""
    O = oracle_lib
    d0, d1 = 1.0, 0.01
    times = [0.0, 0.0, 0.0] + [0.5] * 6
    wl = trace_workload("fcfs", [1], [1], d0, d1, 12, [], times, [0] * 9)
    r = O.run_one(wl, 0, 0, 3, btrace_cap=3)
    b0, b1 = r["batches_trace"][:2]
    assert b0["prefills"] == 3 and b0["mem_after"] == 6
    assert b1["prefills"] == 6 and b1["selected"] == 9
    assert b1["tokens"] == 12 and r["peak_mem"] == 12
    assert b1["completions"] == 3 and b1["mem_after"] == 12


def test_nested_full_prefix_batch_is_mpi(oracle_lib):
    """With segments (1, 2) and thresholds (4, 2) the steady full prefix batch
    processes 4 prefills, 4 stage-1 prompts and 2 boundary prompts; its tokens
    equal M^pi = sum_k n_k (l + sbar_k) delta_k (boundary prompts are processed
    at stage r_1 + 1)."""
    O = oracle_lib
    d1 = 0.01
    d0 = 1.0 - 12.0 * d1
    n = [4, 2]
    times = [1e-4 * i for i in range(200)]
    lengths = [1 + (i % 2) for i in range(200)]   # "Hi" / "Hi there!"
    C = 40
    wl = trace_workload("nested", [1], None, d0, d1, C, n, times, [0] * 200,
                        lengths=lengths, seg_end=[1, 2], out_cap=2)
    r = O.run_one(wl, 0, 0, 12, btrace_cap=12)
    mpi = F.nested_mpi(n, [1, 2], 1)
    toks = [b["tokens"] for b in r["batches_trace"]]
    assert max(toks) == mpi == 18
    assert r["evictions"] == 0 and r["flags"] == 0
    # each request takes exactly L + 1 processing steps (reading A2)
    assert r["batch_tokens_sum"] == sum(
        b["tokens"] for b in r["batches_trace"])


def test_nested_repair_evicts_boundary_first(oracle_lib):
    """With C >= M^pi the restricted repair never needs interior prompts
    (the no-stall property of Nested WAIT's repair rule): an overflowing
    boundary queue is trimmed, most recent first, and memory stays <= C."""
    O = oracle_lib
    d0, d1 = 1.0, 0.001
    n = [2, 1]
    seg_end = [2, 8]
    times = [1e-4 * i for i in range(400)]
    lengths = [8] * 400                    # everyone survives segment 1
    C = 200
    assert F.nested_mpi(n, seg_end, 10) <= C
    wl = trace_workload("nested", [10], None, d0, d1, C, n, times, [0] * 400,
                        lengths=lengths, seg_end=seg_end, out_cap=8)
    r = O.run_one(wl, 0, 0, 80, btrace_cap=80)
    assert r["evictions"] > 0
    assert r["fallback_evictions"] == 0
    assert r["flags"] == 0
    for b in r["batches_trace"]:
        assert b["mem_after"] <= C


def test_nested_fallback_when_capacity_below_mpi(oracle_lib):
    """Below M^pi the boundary queues can run dry; the reading used here then
    evicts interior prompts (counted as fallback evictions) and memory after
    repair still respects C."""
    O = oracle_lib
    d0, d1 = 1.0, 0.001
    times = [1e-4 * i for i in range(400)]
    wl = trace_workload("nested", [10], None, d0, d1, 150, [4, 1], times,
                        [0] * 400, lengths=[8] * 400, seg_end=[2, 8], out_cap=8)
    assert F.nested_mpi([4, 1], [2, 8], 10) > 150
    r = O.run_one(wl, 0, 0, 60, btrace_cap=60)
    assert r["fallback_evictions"] > 0
    for b in r["batches_trace"]:
        assert b["mem_after"] <= 150
