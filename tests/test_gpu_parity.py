"""GPU parity: the HIP path, called through the C ABI, against the oracle.

Counts, admissions, evictions, flags and histograms must be identical; the
fp64 time and latency accumulators must agree within 1e-12 relative (the
two sides perform the same IEEE operations in the same order, so they are
normally bit-identical).
"""
import json
import os

import numpy as np
import pytest

import workloads as W
from tests.parity_util import compare

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module")
def sim():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2504_11320_amd import binding as B
    B.lib()
    return B


def _oracle(jobs, horizon):
    from tests.gpu_util import oracle_results
    return oracle_results(jobs, horizon)


def _check(sim, jobs, horizon, ctx):
    print(f"[gpu] {ctx}: {len(jobs)} jobs, {sum(j.n for j in jobs)} replicas, "
          f"horizon {horizon}", flush=True)
    g = sim.run_batch(jobs, horizon)
    o = _oracle(jobs, horizon)
    st = compare(g, o, ctx)
    print(f"[gpu] {ctx}: ok, fp64 bit-exact {st['f64_bit_exact']}/{st['f64_total']}",
          flush=True)
    return g, o


def test_trace_fcfs_cycle(sim):
    with open(os.path.join(GOLD, "fcfs_cycle_prop3.json")) as f:
        g = json.load(f)
    d1 = g["instance"]["d1"]
    times = [1e-4 * i for i in range(60)]
    wl = W.trace_workload("fcfs", [1], [1], 1.0 - 12 * d1, d1, 12, [], times,
                          [0] * 60, record_capacity=1024)
    res, _ = _check(sim, [W.Job(wl, 0, W.ids(3))], 7, "fcfs trace")
    # 7 batches of the golden trace: 19 completions, 16 evictions
    assert res["completions"][0] == sum(b["completions"] for b in g["batches"])
    assert res["evictions"][0] == sum(b["evicted_after"] for b in g["batches"])


def test_trace_wait_composition(sim):
    d1 = 0.01
    times = [1e-4 * i for i in range(80)]
    wl = W.trace_workload("wait", [1], [1], 1.0 - 12 * d1, d1, 12, [4], times, [0] * 80)
    res, _ = _check(sim, [W.Job(wl, 0, W.ids(2))], 10, "wait trace")
    assert res["peak_mem"][0] == 12 and res["evictions"][0] == 0


def test_config1_parity(sim):
    # the configuration's full horizon: 64 replicas x 10^4 batches, no stop
    res, _ = _check(sim, W.config1(), 10000, "config1 64x10000")
    assert (res["batches"] == 10000).all() and not (res["flags"] & 3).any()


def test_config2_parity_ragged(sim):
    # 70 replicas per rate: the last wave of each job is partial
    jobs = W.config2(replicas=70, rate_index=[0, 15, 31])
    _check(sim, jobs, 3000, "config2 3 rates x70 x3000")


def test_config4_subset_parity(sim):
    jobs = W.config4(replicas=16, grid=16, n_rates=16)
    pick = [jobs[i] for i in (0, 37, 255, 256 * 7 + 100, 256 * 15 + 255)]
    fcfs = [j for j in jobs if j.wl.policy == "fcfs"]
    _check(sim, pick + [fcfs[0], fcfs[8], fcfs[15]], 3000, "config4 subset + FCFS")


def test_resume_equals_one_shot(sim):
    jobs = W.config2(replicas=64, rate_index=[5, 30])
    one = sim.run_batch(jobs, 2500)
    s = sim.Simulation(jobs)
    s.prepare()
    s.advance(1000, resume=False)
    s.advance(1, resume=True)
    s.advance(1499, resume=True)
    two = s.results()
    for k in one:
        assert np.array_equal(one[k], two[k]), k


def test_replica_independence(sim):
    """A replica's outputs depend only on (model, policy, seed, replica id,
    horizon): splitting or reordering jobs changes nothing."""
    base = W.config2(replicas=40, rate_index=[20])[0]
    r1 = sim.run_batch([base], 1500)
    perm = np.array(base.replica_ids[::-1])
    a = W.Job(base.wl, base.seed, perm[:13])
    b = W.Job(base.wl, base.seed, perm[13:])
    other = W.config1(replicas=5)[0]
    r2 = sim.run_batch([a, other, b], 1500)
    order = list(range(13)) + list(range(18, 18 + 27))
    for k in ("batches", "arrivals", "completions", "evictions", "t_end", "lat_area"):
        got = r2[k][order]
        assert np.array_equal(got, r1[k][::-1]), k


def test_edge_cases(sim):
    # horizon 0: nothing happens
    jobs = W.config2(replicas=3, rate_index=[1])
    res = sim.run_batch(jobs, 0)
    assert not np.any(res["batches"]) and not np.any(res["t_end"])
    # a type that never arrives, and a system that can never start
    wl = W.config2(replicas=1, rate_index=[10])[0].wl
    wl.lam = [wl.lam[0], 0.0, wl.lam[2]]
    _check(sim, [W.Job(wl, 0, W.ids(5))], 1500, "zero-rate type")
    wl2 = W.config2(replicas=1, rate_index=[10])[0].wl
    wl2.lam = [0.0, 0.0, 0.0]
    res, _ = _check(sim, [W.Job(wl2, 0, W.ids(2))], 10, "no arrivals (stall)")
    assert np.all(res["flags"] == 2)
    # tiny queue capacity: replicas stop with the capacity flag, counts exact
    wl3 = W.config1()[0].wl
    wl3.record_capacity = 16
    res, _ = _check(sim, [W.Job(wl3, 0, W.ids(64))], 500, "queue capacity")
    assert np.all(res["flags"] & 1)
    # single type, large threshold (long idle accumulation)
    wl4 = W.Workload(prompt_len=[64], lam=[0.05], d0=2.0, d1=0.001, C=5000,
                     policy="wait", n=[40], out_len=[30],
                     hist_edges=W.default_edges(2.0, 100))
    _check(sim, [W.Job(wl4, 7, W.ids(65, start=1000))], 400, "m=1 n=40")
    # FCFS with an admission reserve
    wl5 = [j for j in W.config4(replicas=1, grid=1, n_rates=4) if j.wl.policy == "fcfs"][2].wl
    wl5.reserve = 0.01
    _check(sim, [W.Job(wl5, 3, W.ids(33))], 2000, "fcfs reserve 1%")
    # a job with no replicas between two others; one replica per job
    base = W.config2(replicas=1, rate_index=[7])[0].wl
    empty = W.Job(base, 0, W.ids(0))
    res, _ = _check(sim, [W.Job(base, 0, W.ids(1)), empty, W.Job(wl5, 3, W.ids(1, start=9))],
                    1500, "empty job, single replicas")
    assert len(res["batches"]) == 2
    # no replicas at all is invalid
    with pytest.raises(sim.WaitSimError):
        sim.run_batch([empty], 10)


def test_histogram_edge_sets(sim):
    """Bins through the bucket index equal the oracle's count of edges <= the
    latency for unusual edge sets: negative and zero edges, a span of
    hundreds of binades, many edges in one binade, one edge, none."""
    base = W.config2(replicas=1, rate_index=[12])[0].wl
    sets = [
        [-5.0, -1.0, 0.0, 1e-300, 1e-3, 7.5, 1e300],
        list(np.linspace(14.0, 16.0, 255)),
        [100.0],
        [],
        [-1.0],
        list(np.geomspace(1e-200, 1e200, 255)),
    ]
    jobs = []
    for i, e in enumerate(sets):
        wl = W.Workload(**{**base.__dict__, "hist_edges": np.asarray(e, dtype=np.float64)})
        jobs.append(W.Job(wl, 0, W.ids(40, start=100 * i)))
    _check(sim, jobs, 2500, "histogram edge sets")


@pytest.mark.slow
def test_config2_full_size_sampled(sim):
    """The benchmark's launch: 32 rates x 1024 replicas x 1e5 batches in one
    call; sampled replicas are recomputed one by one by the oracle."""
    from oracle import oracle as O
    jobs = W.config2()
    print("[gpu] config2 full size", flush=True)
    g = sim.run_batch(jobs, 100000)
    assert np.all(g["batches"] == 100000) and not np.any(g["flags"])
    picks = [(ri, rid) for ri in (0, 9, 19, 31) for rid in (0, 1023)]
    per = []
    for ri, rid in picks:
        job = W.Job(jobs[ri].wl, 0, np.array([rid], dtype=np.uint32))
        per.append((ri * 1024 + rid, job))
    outs = [O.run_job(j, 100000, threads=1) for _, j in per]
    o = {k: np.concatenate([x[k] for x in outs]) for k in outs[0]}
    idx = np.array([i for i, _ in per])
    gsub = {k: v[idx] for k, v in g.items()}
    st = compare(gsub, o, "config2 full-size sample")
    print(f"[gpu] config2 full size sample ok, bit-exact fp64 {st}", flush=True)


def test_rate_sweep_stability_point(sim):
    """The Llama-shaped WAIT sweep read with the analysis helpers: completion
    rates follow the arrival rates at low load and fall behind past the
    stability point, which lies inside the swept span (0.5-1.2 Lambda*)."""
    from paper_2504_11320_amd import analysis as A
    jobs = W.config2(replicas=64, n_rates=8)
    res = sim.run_batch(jobs, 20000)
    s = A.summarize(res)
    means = A.job_means(s["completion_rate"], [j.n for j in jobs])
    rates = [sum(j.wl.lam) for j in jobs]
    comp = [m for m, _ in means]
    lam_hat = A.lambda_hat(rates, comp, tol=0.05)
    print(f"[gpu] sweep: lambda_hat / Lambda* = {lam_hat / W.LAM_STAR_C2:.3f}", flush=True)
    assert rates[0] <= lam_hat < rates[-1]
    assert comp[0] >= 0.95 * rates[0] and comp[-1] < 0.95 * rates[-1]


def test_checkpoint_restore(sim):
    """A workspace copy taken between calls is a checkpoint: restored into a
    new Simulation of the same jobs (through host memory) and resumed, it ends
    where the original run ends, bit for bit, for every policy."""
    B = sim
    from tests.test_gpu_random import random_workload
    rng = np.random.default_rng(99)
    jobs = [W.Job(random_workload(rng), 3, W.ids(9)) for _ in range(8)]
    ref = B.run_batch(jobs, 1000)
    a = B.Simulation(jobs)
    a.prepare()
    a.advance(400)
    ck = a.checkpoint(to_host=True)
    b = B.Simulation(jobs)
    b.restore(ck)
    b.advance(600, resume=True)
    got = b.results()
    for k in ref:
        assert np.array_equal(ref[k], got[k]), k
