"""Host logic of bench.py (no GPU): the operation and byte models behind the
roofline figures, the thinning candidate ratio, the profile-summary lookup and
the refusal of more than one GPU."""
import os
import re
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import workloads as W  # noqa: E402


def test_op_model_constants():
    c = bench.op_model(3)
    # Philox4x32-10 (10 rounds of 2 wide multiplies at 4, 4 xor, 2 adds) +
    # uniform + ln + gap = 214 per draw, + 12 bookkeeping + 2m
    assert c["arrival"] == 140 + 10 + 50 + 14 + 12 + 2 * 3
    assert c["batch"] == 24 + 6 * 3
    assert c["completion"] == 35
    assert c["eviction"] == 14 + 3 * 3
    assert c["idle"] == 15 + 4 * 3
    # a 2048-entry CDF row adds 2 ops per halving step (11 steps)
    assert bench.op_model(3, cdf_cap=2048)["arrival"] - c["arrival"] == 22
    # a profile of 25 points: search of 5 halvings at 3 ops + 24 per candidate
    tv = bench.op_model(3, rate_pts=25, cand_per_arrival=1.5)
    assert tv["arrival"] == pytest.approx(1.5 * (214 + 15 + 24) + 12 + 6)


def test_algorithmic_counts_are_linear_in_events():
    res = {k: np.array([v]) for k, v in dict(batches=1000, arrivals=590, completions=550,
                                              evictions=1780, idle_waits=80).items()}
    c = bench.op_model(3)
    want = (1000 * c["batch"] + 590 * c["arrival"] + 550 * c["completion"]
            + 1780 * c["eviction"] + 80 * c["idle"])
    assert bench.algorithmic_ops(res, 3) == pytest.approx(want)
    # the benchmark's event mix gives about 241 lane-operations per batch
    assert 235 < want / 1000 < 245
    # record traffic: 32 bytes per arrival and per completion
    assert bench.algorithmic_bytes(res) == 32 * (590 + 550)


def test_chunks_cover_the_horizon():
    for h, k in ((1000000, 20), (1000000, 3), (10000, 7), (5, 5)):
        c = bench.chunks(h, k)
        assert len(c) == k and sum(c) == h and max(c) - min(c) <= 1


def test_baseline_threads_follow_the_allotment(monkeypatch):
    monkeypatch.setenv("OMP_NUM_THREADS", "3")
    assert bench.baseline_threads() == min(3, bench.host_cpu()["allowed"])
    monkeypatch.delenv("OMP_NUM_THREADS")
    assert 1 <= bench.baseline_threads() <= 16
    cpu = bench.host_cpu()
    assert cpu["nproc"] >= cpu["allowed"] >= 1


def test_candidates_per_arrival():
    base = W.config2(replicas=4, rate_index=[3])[0].wl
    assert bench.candidates_per_arrival([W.Job(base, 0, W.ids(4))]) == 1.0
    # a triangle 0 -> 2 -> 0: mean 1, bound 2, for every type
    tri = W.with_profile(base, [0.0, 1.0, 2.0], np.tile([0.0, 2.0, 0.0], (base.m, 1)))
    assert bench.candidates_per_arrival([W.Job(tri, 0, W.ids(4))]) == pytest.approx(2.0)


def test_profile_summary_lookup(monkeypatch):
    path = os.path.join(ROOT, "profiles", bench.PROFILES["nested-heavytail"][0] + "_hbm.md")
    txt = open(path).read()
    h = re.search(r"source_sha256_16:\s*([0-9a-f]+)", txt).group(1)
    b = float(re.search(r"hbm_bytes_per_replica_iteration:\s*([0-9.eE+]+)", txt).group(1))
    got = bench.traffic_from_profile("nested-heavytail", 1000.0)
    if h == bench.source_hash("nested-heavytail"):
        assert got == pytest.approx(1000.0 * b)
    else:
        assert got is None
    # a summary taken on other sources is not used
    monkeypatch.setattr(bench, "source_hash", lambda workload="wait-llama": "0" * 16)
    assert bench.traffic_from_profile("nested-heavytail", 1.0) is None
    assert bench.traffic_from_profile("no-such-workload", 1.0) is None


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr
    assert p.stdout.strip() == ""


def test_every_workload_runs_on_the_oracle(oracle_lib):
    """Each workload bench.py can time builds its jobs, the policy label and
    the CPU-baseline job picks are consistent with them, and one replica of
    each sampled job runs 50 batches on the oracle without a flag."""
    from oracle import oracle as O
    table = bench._workloads()
    assert next(iter(table)) == "nested-heavytail"
    for name, (desc, build, horizon, policy, picks, cpu_reps) in table.items():
        assert cpu_reps >= 1, name
        jobs = build(4)
        assert desc and horizon > 0, name
        assert all(0 <= p < len(jobs) for p in picks), name
        pols = {j.wl.policy for j in jobs}
        assert pols <= set(policy.split("+")), (name, pols, policy)
        for p in picks:
            j = jobs[p]
            r = O.run_job(W.Job(j.wl, j.seed, j.replica_ids[:1]), 50)
            assert r["batches"][0] == 50 and r["flags"][0] == 0, (name, p)
