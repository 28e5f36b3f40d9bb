"""GPU parity at the library's size limits and across wavefront layouts.

* Maximum model sizes against the oracle: 8 request types for WAIT and FCFS,
  16 types and 16 segments for Nested WAIT, 255 histogram edges.
* Launches large enough that the host packs 16 or 32 replicas per wavefront
  (known-length kernels with up to 4 types stop at 32 and add wavefronts;
  64 per wavefront is covered with 8 types in test_gpu_max_sizes.py): a
  replica's outputs depend only on (model, policy, seed, replica id,
  horizon), so the same replicas run alone (8 per wavefront) must give
  bit-identical results.
"""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import check, sim_module

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    return sim_module()


def _types(rng, m):
    l = [int(x) for x in rng.integers(4, 200, m)]
    lam = [float(x) for x in rng.uniform(0.002, 0.02, m)]
    return l, lam


def test_eight_types_wait_and_fcfs(B):
    rng = np.random.default_rng(16)
    l, lam = _types(rng, 8)
    lp = [int(x) for x in rng.integers(1, 64, 8)]
    C = 4 * max(a + b for a, b in zip(l, lp)) * 4
    edges = W.default_edges(5.0, 255)
    wait = W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=C, policy="wait",
                      n=[int(x) for x in rng.integers(1, 4, 8)], out_len=lp,
                      hist_edges=edges, record_capacity=1 << 12)
    fcfs = W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=C, policy="fcfs", n=[],
                      out_len=lp, reserve=0.01, hist_edges=edges, record_capacity=1 << 12)
    jobs = [W.Job(wait, 11, W.ids(37)), W.Job(fcfs, 12, W.ids(29, start=500))]
    check(B, jobs, 1200, "8 types, WAIT and FCFS, 255 edges")


def test_sixteen_segments_nested(B):
    rng = np.random.default_rng(1616)
    l, lam = _types(rng, 16)
    cap = 64
    seg_end = list(range(4, 65, 4))            # 16 segments
    cdf = np.stack([W.geometric_cdf_table(float(rng.uniform(3.0, 40.0)), cap)
                    for _ in range(16)])
    n = [int(x) for x in rng.integers(1, 3, 16)]
    wl = W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=8000, policy="nested", n=n,
                    out_cap=cap, out_cdf=cdf, seg_end=seg_end,
                    hist_edges=W.default_edges(5.0, 255), record_capacity=1 << 12)
    check(B, [W.Job(wl, 5, W.ids(41))], 1000, "nested, 16 types x 16 segments")


def _subset_equal(B, jobs, horizon, picks, ctx):
    big = B.run_batch(jobs, horizon)
    starts = np.cumsum([0] + [j.n for j in jobs])
    small_jobs = [W.Job(jobs[ji].wl, jobs[ji].seed,
                        np.asarray(jobs[ji].replica_ids[a:b], dtype=np.uint32))
                  for ji, a, b in picks]
    small = B.run_batch(small_jobs, horizon)
    idx = np.concatenate([np.arange(starts[ji] + a, starts[ji] + b) for ji, a, b in picks])
    for k in big:
        assert np.array_equal(big[k][idx], small[k]), (ctx, k)
    print(f"[gpu] {ctx}: {len(idx)} replicas identical to a separate launch", flush=True)


@pytest.mark.parametrize("reps", [512, 1024, 2048])   # 16, 32, 32 (2,048 wavefronts)
def test_wait_layouts_agree(B, reps):
    jobs = W.config2(replicas=reps)
    _subset_equal(B, jobs, 400, [(0, 0, 33), (17, reps - 40, reps), (31, 5, 9)],
                  f"WAIT, {32 * reps} replicas")


@pytest.mark.parametrize("reps", [512, 1024])         # 16, 32 per wavefront
def test_nested_layouts_agree(B, reps):
    jobs = W.config3(replicas=reps)
    _subset_equal(B, jobs, 300, [(0, 0, 33), (20, reps - 40, reps)],
                  f"Nested WAIT, {32 * reps} replicas")


def test_sixteen_types_wait_and_fcfs(B):
    """16 request types under WAIT and FCFS (thresholds up to 3, 255 edges),
    37 + 29 replicas: the 16-slot known-length kernel at 32 replicas per
    wavefront, against the oracle."""
    rng = np.random.default_rng(16)
    l, lam = _types(rng, 16)
    lp = [int(x) for x in rng.integers(1, 64, 16)]
    C = 4 * max(a + b for a, b in zip(l, lp)) * 4
    edges = W.default_edges(5.0, 255)
    wait = W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=C, policy="wait",
                      n=[int(x) for x in rng.integers(1, 4, 16)], out_len=lp,
                      hist_edges=edges, record_capacity=1 << 12)
    fcfs = W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=C, policy="fcfs", n=[],
                      out_len=lp, reserve=0.01, hist_edges=edges, record_capacity=1 << 12)
    jobs = [W.Job(wait, 11, W.ids(37)), W.Job(fcfs, 12, W.ids(29, start=500))]
    check(B, jobs, 1200, "16 types, WAIT and FCFS, 255 edges")


def test_many_types_nested_and_fcfs(B):
    """Beyond 16 types: Nested WAIT with 40 types and 12 segments (lane groups
    of 64) and with 24 types (groups of 32), FCFS with 64 types, known and
    drawn output lengths (the kernel for per-request lengths), against the
    oracle."""
    rng = np.random.default_rng(64)
    jobs = []
    for m, nseg in ((40, 12), (24, 5)):
        l, lam = _types(rng, m)
        cap = 96
        cuts = sorted(rng.choice(np.arange(1, cap), size=nseg - 1, replace=False).tolist())
        cdf = np.stack([W.geometric_cdf_table(float(rng.uniform(2.0, 40.0)), cap)
                        for _ in range(m)])
        C = int((max(l) + cap) * 3)
        wl = W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=C, policy="nested",
                        n=[int(x) for x in rng.integers(1, 3, nseg)], out_cap=cap,
                        out_cdf=cdf, seg_end=[int(c) for c in cuts] + [cap],
                        hist_edges=W.default_edges(5.0, 128), record_capacity=1 << 12)
        jobs.append(W.Job(wl, 21, W.ids(6)))
    l, lam = _types(rng, 64)
    lp = [int(x) for x in rng.integers(1, 48, 64)]
    C = 3 * max(a + b for a, b in zip(l, lp))
    known = W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=C, policy="fcfs", n=[],
                       out_len=lp, reserve=0.01, hist_edges=W.default_edges(5.0, 128),
                       record_capacity=1 << 12)
    cdf = np.stack([W.geometric_cdf_table(float(rng.uniform(2.0, 30.0)), 48) for _ in range(64)])
    drawn = W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=C, policy="fcfs", n=[],
                       out_cap=48, out_cdf=cdf, hist_edges=W.default_edges(5.0, 128),
                       record_capacity=1 << 12)
    jobs += [W.Job(known, 22, W.ids(9)), W.Job(drawn, 23, W.ids(9))]
    g, _ = check(B, jobs, 1500, "40/24-type Nested WAIT, 64-type FCFS")
    assert g["evictions"].sum() > 0


def test_many_types_wait(B):
    """WAIT beyond 16 types (per-type state in LDS columns): 20 and 64 types,
    thresholds up to 3, tight memory; WAIT-no-wait with 24 types; per-stage
    caps on 20 types; an arrival list with 40 types; against the oracle."""
    rng = np.random.default_rng(65)
    jobs = []
    for m, pol in ((20, "wait"), (64, "wait"), (24, "wait-nowait")):
        l, lam = _types(rng, m)
        lp = [int(x) for x in rng.integers(1, 40, m)]
        C = int(max(a + b for a, b in zip(l, lp)) * rng.uniform(2.0, 4.0))
        wl = W.Workload(prompt_len=l, lam=[x * 3 for x in lam], d0=5.0, d1=0.01, C=C,
                        policy=pol, n=[int(x) for x in rng.integers(1, 4, m)], out_len=lp,
                        hist_edges=W.default_edges(5.0, 128), record_capacity=1 << 12)
        jobs.append(W.Job(wl, 31, W.ids(10)))
    l, lam = _types(rng, 20)
    lp = [int(x) for x in rng.integers(1, 30, 20)]
    caps, n = [], []
    for lpj in lp:
        seg = [2] * int(rng.integers(0, lpj + 1)) + [1] * (lpj + 1)
        seg = seg[:lpj + 1]
        caps += seg
        n.append(max(seg))
    C = int(max(a + b for a, b in zip(l, lp)) * 3)
    jobs.append(W.Job(W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=C, policy="wait",
                                 n=n, out_len=lp, stage_caps=caps,
                                 hist_edges=W.default_edges(5.0, 128), record_capacity=1 << 12),
                      32, W.ids(10)))
    g, _ = check(B, jobs, 1500, "WAIT with 20-64 types")
    assert g["evictions"].sum() > 0
    times = np.sort(rng.uniform(0.0, 400.0, 600))
    types = rng.integers(0, 40, 600)
    lp = [int(x) for x in rng.integers(1, 12, 40)]
    wl = W.trace_workload("wait", [int(x) for x in rng.integers(1, 20, 40)], lp, 1.0, 0.01, 300,
                          [int(x) for x in rng.integers(1, 3, 40)], times, types,
                          record_capacity=1 << 10)
    check(B, [W.Job(wl, 0, W.ids(3))], 400, "WAIT, 40 types, arrival list")
