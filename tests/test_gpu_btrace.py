"""Per-batch traces from the GPU (wait_sim_advance_traced) against the
oracle's, batch by batch: launch time and duration (fp64 within 1e-12
relative), tokens, prefill processings, selected prompts, completions,
evictions before and after the batch, memory, waiting and resident prompts
(exact), for every policy, with chunked prefill and time-varying rates, and
across a resumed call."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import sim_module

pytestmark = pytest.mark.gpu

INT_F = ("tokens", "prefills", "selected", "completions", "evict_pre", "evict_post",
         "mem_after", "waiting_after", "resident_after", "mplus")


@pytest.fixture(scope="module")
def B():
    return sim_module()


def _models():
    from tests.test_gpu_random import random_workload
    rng = np.random.default_rng(123)
    out = []
    for pol in ("wait", "wait-nowait", "fcfs", "nested"):
        k = 0
        while k < 2:
            wl = random_workload(rng)
            if wl.policy != pol:
                continue
            out.append(wl)
            k += 1
    ch = random_workload(np.random.default_rng(7))
    while ch.policy != "fcfs":
        ch = random_workload(rng)
    ch.chunk = 9
    out.append(ch)
    llama = W.config2(replicas=1, rate_index=[28])[0].wl
    rt, rf = W.diurnal_profile(3, 4.0e6, points=9)
    out.append(W.with_profile(llama, rt, rf))
    out.append(W.config3(replicas=1, rate_index=[31])[0].wl)
    return out


def _compare(g, o, nb, ctx):
    for b in range(nb):
        rec = o[b]
        for f in INT_F:
            assert g[b][f] == rec[f], (ctx, b, f, g[b][f], rec[f])
        for f in ("t_launch", "tau"):
            x, y = float(g[b][f]), rec[f]
            assert abs(x - y) <= 1e-12 * max(abs(y), 1e-300), (ctx, b, f, x, y)


def test_traces_match_the_oracle(B):
    from oracle import oracle as O
    H = 300
    models = _models()
    jobs = [W.Job(wl, 11 + i, W.ids(5)) for i, wl in enumerate(models)]
    sim = B.Simulation(jobs)
    sim.prepare()
    tr = sim.advance_traced(H, H)
    res = sim.results()
    start = 0
    for ji, job in enumerate(jobs):
        for x in (0, 4):
            r = start + x
            o = O.run_one(job.wl, job.seed, int(job.replica_ids[x]), H, btrace_cap=H)
            nb = int(res["batches"][r])
            assert nb == o["batches"]
            _compare(tr[r], o["batches_trace"], nb, f"job {ji} ({job.wl.policy}) replica {x}")
        start += job.n
    print(f"[gpu] per-batch traces: {len(jobs)} jobs x 2 replicas x {H} batches match",
          flush=True)


def test_trace_across_resume(B):
    models = _models()[:4]
    jobs = [W.Job(wl, 5, W.ids(3)) for wl in models]
    one = B.Simulation(jobs)
    one.prepare()
    t1 = one.advance_traced(200, 200)
    two = B.Simulation(jobs)
    two.prepare()
    a = two.advance_traced(120, 200)
    b = two.advance_traced(80, 200, resume=True)
    merged = a.copy()
    merged[:, 120:] = b[:, 120:]
    assert np.array_equal(t1.view(np.uint8), merged.view(np.uint8))
    # the untraced advance gives the same results
    plain = B.run_batch(jobs, 200)
    r1 = one.results()
    for k in plain:
        assert np.array_equal(plain[k], r1[k]), k


def test_prelaunch_repair_hand_traces(B):
    """The hand-traced instances of Nested WAIT's pre-launch repair
    (golden/nested_prelaunch_repair.json: Q+ before and after the repair,
    boundary LIFO across queues, interior fallback, OVERFLOW) replayed on
    the GPU: every batch record equals the hand trace, and the results
    equal the oracle's."""
    from oracle import oracle as O
    from tests.test_oracle_nested_prelaunch import _instances, _workload
    inst = _instances()
    names = sorted(inst)
    jobs = [W.Job(_workload(inst[n]), 0, W.ids(3)) for n in names]
    H = max(g["horizon"] for g in inst.values()) + 2
    sim = B.Simulation(jobs)
    sim.prepare()
    tr = sim.advance_traced(H, H)
    res = sim.results()
    start = 0
    for n, job in zip(names, jobs):
        g = inst[n]
        h = g["horizon"]
        o = O.run_one(job.wl, 0, 0, H, btrace_cap=H)
        for x in range(job.n):
            r = start + x
            nb = int(res["batches"][r])
            assert nb == o["batches"], (n, x)
            _compare(tr[r], o["batches_trace"], nb, f"{n} replica {x}")
            for b, want in enumerate(g["batches"][:h]):
                for f in INT_F[:-1]:
                    assert tr[r][b][f] == want[f], (n, b, f)
                assert tr[r][b]["mplus"] == want["mplus_after"], (n, b)
            assert bool(res["flags"][r] & B.WS_FLAG_OVERFLOW) == g["final"]["overflow"], n
            for f in ("evictions", "fallback_evictions", "evicted_tokens"):
                assert res[f][r] == o[f], (n, f)
        start += job.n
    print(f"[gpu] pre-launch repair hand traces: {len(names)} instances match", flush=True)
