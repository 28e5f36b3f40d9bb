"""Invariants and statistical statements the paper fixes, checked on the oracle.

* request conservation: arrivals = completions + waiting + resident;
* Little's law on the sample path: the accumulated area of N(t) equals the sum
  of per-request censored times in system (Section 2.4, censored delays), and
  the same for the time to first token;
* busy time = batches d0 + d1 sum(tokens) (eq. time_consump);
* WAIT's resident-memory invariant: memory never exceeds M^pi, so no eviction
  when M^pi <= C (lemma on GPU-resident memory in the proof of Theorem 1);
* Proposition 2: completed decode tokens never exceed those that arrived;
* convergence of WAIT to the fluid throughput on an integer instance
  (Theorem 1), the FCFS throughput gap (Proposition 3), instability when
  d1 A >= 1 (Proposition 1), and Nested WAIT's eviction bound (Theorem 2).
"""
import math

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle import fluid as F
from workloads import Workload, default_edges, geometric_cdf_table


def _policy_workloads(draw):
    policy = draw(st.sampled_from(["wait", "fcfs", "nested"]))
    m = draw(st.integers(1, 3))
    l = [draw(st.integers(1, 12)) for _ in range(m)]
    lam = [draw(st.floats(0.05, 1.5)) for _ in range(m)]
    d0 = draw(st.floats(0.2, 3.0))
    d1 = draw(st.floats(0.0, 0.05))
    if policy == "nested":
        cap = draw(st.integers(2, 10))
        nseg = draw(st.integers(1, min(3, cap)))
        cuts = sorted(draw(st.sets(st.integers(1, cap - 1), min_size=nseg - 1,
                                   max_size=nseg - 1)))
        seg_end = list(cuts) + [cap]
        n = [draw(st.integers(1, 4)) for _ in range(nseg)]
        cdf = np.stack([geometric_cdf_table(draw(st.floats(1.2, 6.0)), cap)
                        for _ in range(m)])
        Cmin = max(l) + cap
        C = draw(st.integers(Cmin, Cmin * 8))
        return Workload(prompt_len=l, lam=lam, d0=d0, d1=d1, C=C, policy=policy,
                        n=n, out_cap=cap, out_cdf=cdf, seg_end=seg_end,
                        hist_edges=default_edges(d0, 48), record_capacity=1 << 20)
    lp = [draw(st.integers(1, 8)) for _ in range(m)]
    n = [draw(st.integers(1, 4)) for _ in range(m)] if policy == "wait" else []
    Cmin = max(a + b for a, b in zip(l, lp))
    C = draw(st.integers(Cmin, Cmin * 8))
    return Workload(prompt_len=l, lam=lam, d0=d0, d1=d1, C=C, policy=policy, n=n,
                    out_len=lp, hist_edges=default_edges(d0, 48),
                    record_capacity=1 << 20)


@settings(max_examples=60, deadline=None,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(st.data())
def test_sample_path_identities(oracle_lib, data):
    O = oracle_lib
    wl = _policy_workloads(data.draw)
    horizon = data.draw(st.integers(1, 300))
    rid = data.draw(st.integers(0, 1000))
    r = O.run_one(wl, 11, rid, horizon, rlog_cap=200000)
    T = r["t_end"]
    n_arr = r["arrivals"]
    assert r["flags"] & O.FLAG_CAPACITY == 0
    # conservation
    assert n_arr == r["completions"] + r["waiting_end"] + r["resident_end"]
    # Little's law on the path: area of N = sum of censored times in system
    a = r["req_arr"][:n_arr]
    c = r["req_done"][:n_arr]
    f = r["req_first"][:n_arr]
    assert np.all(a <= T)
    lat = np.where(c >= 0, c, T) - a
    ttft = np.where(f >= 0, f, T) - a
    scale = max(1.0, abs(r["lat_area"]))
    assert abs(math.fsum(lat) - r["lat_area"]) <= 1e-10 * scale
    assert abs(math.fsum(ttft) - r["ttft_area"]) <= 1e-10 * max(1.0, abs(r["ttft_area"]))
    done = c >= 0
    assert done.sum() == r["completions"]
    assert abs(math.fsum((c - a)[done]) - r["lat_completed_sum"]) <= 1e-10 * max(
        1.0, r["lat_completed_sum"])
    assert r["hist"].sum() == r["completions"]
    # latency histogram (reading A21): bin = number of edges <= latency, here by
    # numpy's binary search over every completed request's latency
    edges = np.asarray(wl.hist_edges, dtype=np.float64)
    bins = np.searchsorted(edges, (c - a)[done], side="right")
    assert np.array_equal(np.bincount(bins, minlength=len(edges) + 1), r["hist"])
    # first token is produced no later than completion
    assert np.all(f[done] <= c[done]) and np.all(f[done] >= 0)
    # iteration time identity
    busy = r["batches"] * wl.d0 + wl.d1 * r["batch_tokens_sum"]
    assert abs(busy - r["busy_time"]) <= 1e-9 * max(1.0, busy)
    assert r["busy_time"] <= T * (1 + 1e-12)
    # Proposition 2 pathwise: completed tokens <= decode tokens that arrived
    if wl.out_len is not None and wl.trace is None:
        assert r["completed_tokens"] <= n_arr * max(wl.out_len)
    assert r["batches"] <= horizon


@settings(max_examples=40, deadline=None)
@given(st.data())
def test_wait_memory_invariant(oracle_lib, data):
    """Memory never exceeds M^pi under WAIT, hence no eviction if M^pi <= C."""
    O = oracle_lib
    m = data.draw(st.integers(1, 3))
    l = [data.draw(st.integers(1, 20)) for _ in range(m)]
    lp = [data.draw(st.integers(1, 10)) for _ in range(m)]
    n = [data.draw(st.integers(1, 5)) for _ in range(m)]
    lam = [data.draw(st.floats(0.1, 3.0)) for _ in range(m)]
    mpi = F.wait_mpi(n, l, lp)
    C = int(mpi) + data.draw(st.integers(0, 10))
    wl = Workload(prompt_len=l, lam=lam, d0=1.0, d1=0.01, C=C, policy="wait", n=n,
                  out_len=lp, record_capacity=1 << 20)
    r = O.run(wl, 3, np.arange(4, dtype=np.uint32), 400, threads=4)
    assert np.all(r["evictions"] == 0)
    assert np.all(r["peak_mem"] <= mpi)


def test_wait_approaches_fluid_throughput(oracle_lib):
    """Theorem 1 on the integer instance (2,2),(1,4), lam (3,2), d0 0.43,
    d1 0.01: n* = (3, 2), M* = M^pi = C = 57, fluid throughput 14; with slack
    (rates x0.9) the throughput is the offered load and nothing is evicted."""
    O = oracle_lib
    for scale, tol in ((1.0, 0.03), (0.9, 0.01)):
        lam = [3.0 * scale, 2.0 * scale]
        wl = Workload(prompt_len=[2, 1], lam=lam, d0=0.43, d1=0.01, C=57,
                      policy="wait", n=[3, 2], out_len=[2, 4],
                      record_capacity=1 << 20)
        r = O.run(wl, 0, np.arange(32, dtype=np.uint32), 20000)
        thr = r["completed_tokens"].sum() / r["t_end"].sum()
        target = F.fluid([2, 1], [2, 4], lam, 0.43, 0.01)["throughput"]
        assert abs(thr - target) / target < tol, (scale, thr, target)
        assert r["evictions"].sum() == 0
        assert np.all(r["peak_mem"] <= 57)
        if scale == 1.0:
            # mean batch memory at launch approaches M* = 57
            assert r["mem_area"].sum() / r["busy_time"].sum() > 0.9 * 57


def test_fcfs_throughput_gap_vs_wait(oracle_lib):
    """Proposition 3's instance with Poisson arrivals: FCFS falls short of the
    fluid throughput 4 by a constant, WAIT with n* = 4 does not."""
    O = oracle_lib
    d1 = 0.01
    d0 = 1.0 - 12 * d1
    ids = np.arange(64, dtype=np.uint32)
    common = dict(prompt_len=[1], lam=[4.0], d0=d0, d1=d1, C=12, out_len=[1],
                  record_capacity=1 << 20)
    rf = O.run(Workload(policy="fcfs", n=[], **common), 0, ids, 4000)
    rw = O.run(Workload(policy="wait", n=[4], **common), 0, ids, 4000)
    thr_f = rf["completed_tokens"].sum() / rf["t_end"].sum()
    thr_w = rw["completed_tokens"].sum() / rw["t_end"].sum()
    assert thr_f < 3.7
    assert thr_w > 3.85
    assert rw["evictions"].sum() == 0 and rf["evictions"].sum() > 0


def test_prop1_latency_grows_linearly(oracle_lib):
    """Configuration 1 has d1 A = 2.08 >= 1: mean censored latency grows in
    proportion to the horizon."""
    O = oracle_lib
    from workloads import config1
    job = config1(replicas=8)[0]
    ratios = []
    for h in (500, 2000):
        r = O.run_job(job, h)
        mean_lat = r["lat_area"].sum() / r["arrivals"].sum()
        ratios.append(mean_lat / r["t_end"].mean())
    assert min(ratios) > 0.2
    assert abs(ratios[1] - ratios[0]) < 0.15


def test_nested_eviction_probability_bound(oracle_lib):
    """Theorem 2 (segment form): with thresholds meeting the drift conditions
    and C >= M_req for delta = 0.1, the fraction of replicas with any eviction
    is at most delta."""
    O = oracle_lib
    l, seg_end, n = 4, [4, 8], [4, 2]
    # output length 4 w.p. 0.7, 8 w.p. 0.3  ->  p_2 = 0.3 < n2/n1 = 0.5 < 1
    cap = 8
    F_ = [0.0, 0.0, 0.0, 0.7, 0.7, 0.7, 0.7]
    row = np.array([min(0xFFFFFFFF, int(math.floor(x * 2**32))) for x in F_], dtype=np.uint32)
    lam, d0, d1 = 1.0, 1.0, 0.01
    assert d0 + d1 * F.nested_mpi(n, seg_end, l) < n[0] / lam
    horizon = 3000
    zT = horizon * 8.0                  # bound on the simulated time span
    req = F.nested_m_req(n, seg_end, l, [0.3], m=2, zeta_T=zT, d0=d0, delta=0.1)
    C = int(math.ceil(req["Mreq"]))
    wl = Workload(prompt_len=[l], lam=[lam], d0=d0, d1=d1, C=C, policy="nested",
                  n=n, out_cap=cap, out_cdf=row[None, :], seg_end=seg_end,
                  record_capacity=1 << 20)
    r = O.run(wl, 0, np.arange(200, dtype=np.uint32), horizon)
    assert r["t_end"].max() <= zT
    frac = np.mean(r["evictions"] > 0)
    assert frac <= 0.1


def test_histogram_bin_at_an_edge(oracle_lib):
    """Reading A21: a latency equal to an edge counts that edge (bin = number
    of edges <= latency), so it lands in the bin above the edge."""
    import dataclasses
    O = oracle_lib
    # one prompt arriving at 0 under WAIT-no-wait (served while resident), tau = 1 ms:
    # it passes its l'_j + 1 = 4 stages in four batches, latency 4 ms
    base = Workload(prompt_len=[4], lam=[0.0], d0=1.0, d1=0.0, C=1000, policy="wait-nowait",
                    n=[1], out_len=[3], hist_edges=np.array([0.5]), record_capacity=16,
                    trace=(np.array([0.0]), np.array([0], np.int32), np.array([3], np.int32)))
    r = O.run_one(base, 0, 0, 10, rlog_cap=4)
    assert r["completions"] == 1
    lat = r["req_done"][0] - r["req_arr"][0]
    assert lat == 4.0
    for edges, want in (([lat - 0.5, lat, lat + 0.5], 2), ([lat], 1),
                        ([np.nextafter(lat, np.inf)], 0), ([np.nextafter(lat, -np.inf)], 1)):
        wl = dataclasses.replace(base, hist_edges=np.array(edges, dtype=np.float64))
        h = O.run_one(wl, 0, 0, 10)["hist"]
        assert h.sum() == 1 and h[want] == 1, (edges, h)


HIST_MUTATIONS = {
    # an edge equal to the latency not counted
    "strict": ("while (b < c->n_edges && c->edges[b] <= lat) b++;",
               "while (b < c->n_edges && c->edges[b] < lat) b++;"),
    # the index of the last edge <= latency instead of their number
    "last_edge": ("  return b;\n}\n\nstatic void complete(",
                  "  return b > 0 ? b - 1 : 0;\n}\n\nstatic void complete("),
}


def _hist_mismatch(O, library) -> bool:
    """Run the edge-equality case and a random WAIT path through `library`
    and report whether any histogram disagrees with the definition."""
    import dataclasses
    base = Workload(prompt_len=[4], lam=[0.0], d0=1.0, d1=0.0, C=1000, policy="wait-nowait",
                    n=[1], out_len=[3], hist_edges=np.array([4.0]), record_capacity=16,
                    trace=(np.array([0.0]), np.array([0], np.int32), np.array([3], np.int32)))
    h = O.run_one(base, 0, 0, 10, library=library)["hist"]
    if h.sum() != 1 or h[1] != 1:
        return True
    wl = Workload(prompt_len=[16, 40], lam=[0.3, 0.2], d0=2.0, d1=0.01, C=4000, policy="wait",
                  n=[2, 1], out_len=[6, 20], hist_edges=default_edges(2.0, 96),
                  record_capacity=1 << 14)
    r = O.run_one(wl, 3, 5, 400, rlog_cap=1 << 14, library=library)
    a, c = r["req_arr"][:r["arrivals"]], r["req_done"][:r["arrivals"]]
    done = c >= 0
    bins = np.searchsorted(wl.hist_edges, (c - a)[done], side="right")
    return not np.array_equal(np.bincount(bins, minlength=len(wl.hist_edges) + 1), r["hist"])


@pytest.mark.parametrize("name", sorted(HIST_MUTATIONS))
def test_histogram_pins_reject_planted_mistakes(oracle_lib, tmp_path, name):
    import os
    import subprocess
    O = oracle_lib
    assert not _hist_mismatch(O, None)
    src = open(O.SRC).read()
    old, new = HIST_MUTATIONS[name]
    assert src.count(old) == 1, name
    path = tmp_path / f"wait_oracle_{name}.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / f"liboracle_{name}.so"
    subprocess.run(["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math",
                    "-fPIC", "-shared", "-I", os.path.dirname(O.SRC), "-o", str(lib),
                    str(path), "-lpthread", "-lm"], check=True)
    assert _hist_mismatch(O, O.load(str(lib))), name
