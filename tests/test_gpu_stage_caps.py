"""Per-stage caps of Nested WAIT and WAIT (Section 6) on the GPU, against the
oracle.

The hand-traced instance (golden/nested_stage_caps.json) replayed batch by
batch; the two-type p512 mix with the caps that the batch-size cap tl = 30
gives (segment caps 21 and 9 spread over 20 and 30 decode stages); random
models with random caps, tight memory included; uniform caps against the
same jobs without caps (the general and the specialised kernels); a resumed
run through a checkpoint.  WAIT: its hand trace (golden/wait_stage_caps.json),
random capped models with evictions, uniform caps against the specialised
kernel, and the single-type p512d20 workload with the caps of tl = 30.
"""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import check, sim_module

pytestmark = pytest.mark.gpu

INT_F = ("tokens", "prefills", "selected", "completions", "evict_pre", "evict_post",
         "mem_after", "waiting_after", "resident_after", "mplus")


@pytest.fixture(scope="module")
def B():
    return sim_module()


def _spread(total, stages):
    base, extra = divmod(total, stages)
    return [base + 1] * extra + [base] * (stages - extra)


def random_capped(rng):
    """A random Nested WAIT model whose segment caps B_k are spread over the
    segment's decode stages (segment 1 keeps every cap >= 1)."""
    from tests.test_oracle_stage_caps import _random_nested
    wl = _random_nested(rng)
    caps, n, lo = [], [], 0
    for k, e in enumerate(wl.seg_end):
        width = e - lo
        total = int(rng.integers(width if k == 0 else 1, 3 * width + 1))
        seg = _spread(total, width)
        if rng.random() < 0.5:  # the larger caps last
            seg = seg[::-1]
        caps += seg
        n.append(max(seg))
        lo = e
    wl.stage_caps = caps
    wl.n = n
    return wl


def test_hand_trace_on_the_gpu(B):
    from oracle import oracle as O
    from tests.test_oracle_stage_caps import _gold, _workload
    g = _gold()
    job = W.Job(_workload(g), 0, W.ids(3))
    H = g["instance"]["horizon"]
    print(f"[gpu] stage caps hand trace, horizon {H}", flush=True)
    sim = B.Simulation([job])
    sim.prepare()
    tr = sim.advance_traced(H, H)
    res = sim.results()
    o = O.run_one(job.wl, 0, 0, H, btrace_cap=H)
    for r in range(job.n):
        for b, want in enumerate(g["batches"]):
            for f in INT_F:
                assert tr[r][b][f] == want[f], (r, b, f)
            assert float(tr[r][b]["t_launch"]) == want["t_launch"], (r, b)
        for k, v in g["final"].items():
            assert res[k][r] == v, (r, k)
        for k in ("batches", "completions", "idle_waits", "lat_completed_sum", "t_end"):
            assert res[k][r] == o[k], (r, k)


def test_p512_mix_tl30_parity(B):
    jobs = W.config_p512_mix(replicas=64)
    g, _ = check(B, jobs, 3000, "p512 mix tl=30 caps")
    assert (g["batches"] == 3000).all()


def test_random_capped_models(B):
    rng = np.random.default_rng(77)
    jobs = [W.Job(random_capped(rng), 9, W.ids(8)) for _ in range(16)]
    g, _ = check(B, jobs, 1500, "random capped Nested WAIT")
    assert g["evictions"].sum() > 0  # tight memory in some of the models
    # interior (fallback) evictions, back to back and from partly filled
    # cohort rows: the kernel's cached youngest records are exercised
    assert g["fallback_evictions"].sum() > 1000


def test_uniform_caps_equal_the_specialised_kernel(B):
    """Caps equal to n_k everywhere run in the general instantiation and give
    the same results as the jobs without caps."""
    jobs = W.config3(replicas=48, rate_index=[10, 31])
    capped = []
    for j in jobs:
        caps, lo = [], 0
        for e, nk in zip(j.wl.seg_end, j.wl.n):
            caps += [nk] * (e - lo)
            lo = e
        wl = W.Workload(**{**j.wl.__dict__, "stage_caps": caps})
        capped.append(W.Job(wl, j.seed, j.replica_ids))
    a = B.run_batch(jobs, 2000)
    b = B.run_batch(capped, 2000)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_capped_checkpoint_resume(B):
    import torch
    jobs = W.config_p512_mix(replicas=32, rates=[0.022])
    ref = B.Simulation(jobs)
    ref.run_ex(1500)
    want = ref.results()
    a = B.Simulation(jobs)
    out = torch.empty(16 << 20, dtype=torch.uint8, device="cuda")
    used = a.run_ex(600, state_out=out)
    c = B.Simulation(jobs)
    c.run_ex(900, state_in=out[:used].clone())
    got = c.results()
    for k in want:
        assert np.array_equal(want[k], got[k]), k


# ----------------------------------------------------------------- WAIT ----

def random_capped_wait(rng):
    """A random WAIT model whose per-type caps spread a random total over the
    type's l'_j + 1 stages (every cap >= 1)."""
    from tests.test_oracle_stage_caps import _random_wait
    wl = _random_wait(rng)
    caps, n = [], []
    for lpj in wl.out_len:
        width = lpj + 1
        seg = _spread(int(rng.integers(width, 3 * width + 1)), width)
        if rng.random() < 0.5:
            seg = seg[::-1]
        caps += seg
        n.append(max(seg))
    wl.stage_caps = caps
    wl.n = n
    return wl


def test_wait_hand_trace_on_the_gpu(B):
    from oracle import oracle as O
    from tests.test_oracle_stage_caps import _wait_gold, _wait_workload
    g = _wait_gold()
    job = W.Job(_wait_workload(g), 0, W.ids(3))
    H = g["instance"]["horizon"]
    print(f"[gpu] WAIT stage caps hand trace, horizon {H}", flush=True)
    sim = B.Simulation([job])
    sim.prepare()
    tr = sim.advance_traced(H, H)
    res = sim.results()
    o = O.run_one(job.wl, 0, 0, H, btrace_cap=H)
    for r in range(job.n):
        for b, want in enumerate(g["batches"]):
            for f in INT_F[:-1]:
                assert tr[r][b][f] == want[f], (r, b, f)
            assert float(tr[r][b]["t_launch"]) == want["t_launch"], (r, b)
        for k, v in g["final"].items():
            assert res[k][r] == v, (r, k)
        for k in ("batches", "completions", "idle_waits", "lat_completed_sum", "t_end"):
            assert res[k][r] == o[k], (r, k)


def test_wait_random_capped_models(B):
    rng = np.random.default_rng(83)
    jobs = [W.Job(random_capped_wait(rng), 9, W.ids(8)) for _ in range(16)]
    g, _ = check(B, jobs, 1500, "random capped WAIT")
    assert g["evictions"].sum() > 0


def test_wait_uniform_caps_equal_the_specialised_kernel(B):
    jobs = W.config2(replicas=48, rate_index=[10, 31])
    capped = []
    for j in jobs:
        caps = sum(([nj] * (lpj + 1) for nj, lpj in zip(j.wl.n, j.wl.out_len)), [])
        capped.append(W.Job(W.Workload(**{**j.wl.__dict__, "stage_caps": caps}), j.seed,
                            j.replica_ids))
    a = B.run_batch(jobs, 2000)
    b = B.run_batch(capped, 2000)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_wait_p512d20_tl30_parity(B):
    from paper_2504_11320_amd import calibrate as Cal
    caps = Cal.calibrate_wait(30, 20)["stage_caps"]
    jobs = []
    for j in W.config_p512d20(replicas=48)[:7]:  # the WAIT jobs, 0.6-1.0 of the boundary
        wl = W.Workload(**{**j.wl.__dict__, "stage_caps": caps, "n": [max(caps)]})
        jobs.append(W.Job(wl, j.seed, j.replica_ids))
    check(B, jobs, 4000, "p512d20 WAIT, caps of tl=30")
