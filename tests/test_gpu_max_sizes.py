"""The widest instantiations at the library's size limits, in launches large
enough that the host packs the most replicas per wavefront: Nested WAIT with
16 types, 16 segments and 255 histogram edges at 32 replicas per wavefront
(65,536 replicas), with and without a 32-point rate profile; WAIT and FCFS
with 8 types at 64 replicas per wavefront.  Sampled replicas (first, last
and interior wavefronts) are compared with the oracle field by field."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import sim_module
from tests.parity_util import compare

pytestmark = pytest.mark.gpu

R = 65536


def _sampled(B, jobs, H, ctx, picks=(0, 31, 32, 40000, R - 1)):
    from oracle import oracle as O
    g = B.run_batch(jobs, H)
    start = 0
    for job in jobs:
        idx = np.array(picks)
        sub = W.Job(job.wl, job.seed, job.replica_ids[idx])
        o = O.run_job(sub, H)
        gs = {k: v[start + idx] for k, v in g.items()}
        gs["hist"] = gs["hist"][:, :o["hist"].shape[1]]
        compare(gs, o, ctx)
        start += job.n
    print(f"[gpu] {ctx}: sampled replicas match", flush=True)
    return g


def _nested16(rng):
    l = [int(x) for x in rng.integers(4, 60, 16)]
    lam = [float(x) for x in rng.uniform(0.002, 0.01, 16)]
    cap = 64
    cdf = np.stack([W.geometric_cdf_table(float(rng.uniform(3.0, 40.0)), cap)
                    for _ in range(16)])
    return W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=3000, policy="nested",
                      n=[int(x) for x in rng.integers(1, 3, 16)], out_cap=cap, out_cdf=cdf,
                      seg_end=list(range(4, 65, 4)), hist_edges=W.default_edges(5.0, 255),
                      record_capacity=1 << 9)


def test_nested_16x16_at_32_per_wavefront():
    B = sim_module()
    wl = _nested16(np.random.default_rng(1616))
    print(f"[gpu] nested 16x16, {R} replicas", flush=True)
    g = _sampled(B, [W.Job(wl, 7, W.ids(R))], 400, "nested 16 types x 16 segments, 32/wave")
    assert g["arrivals"].min() >= 0 and g["completions"].sum() > 0


def test_nested_16x16_with_profile():
    B = sim_module()
    wl = _nested16(np.random.default_rng(1617))
    rt, rf = W.diurnal_profile(16, 3.0e4, points=32, amp=0.8)
    wl = W.with_profile(wl, rt, rf)
    print(f"[gpu] nested 16x16 with a 32-point profile, {R} replicas", flush=True)
    _sampled(B, [W.Job(wl, 8, W.ids(R))], 400, "nested 16x16, 32-point profile")


def test_wait_and_fcfs_8_types_at_64_per_wavefront():
    B = sim_module()
    rng = np.random.default_rng(88)
    l = [int(x) for x in rng.integers(4, 200, 8)]
    lam = [float(x) for x in rng.uniform(0.002, 0.02, 8)]
    lp = [int(x) for x in rng.integers(1, 64, 8)]
    C = 16 * max(a + b for a, b in zip(l, lp))
    edges = W.default_edges(5.0, 255)
    wait = W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=C, policy="wait",
                      n=[int(x) for x in rng.integers(1, 4, 8)], out_len=lp,
                      hist_edges=edges, record_capacity=1 << 10)
    fcfs = W.Workload(prompt_len=l, lam=lam, d0=5.0, d1=0.01, C=C, policy="fcfs", n=[],
                      out_len=lp, reserve=0.01, hist_edges=edges, record_capacity=1 << 10)
    print(f"[gpu] 8 types, WAIT and FCFS, {R} replicas each", flush=True)
    _sampled(B, [W.Job(wait, 3, W.ids(R)), W.Job(fcfs, 4, W.ids(R))], 600,
             "WAIT and FCFS, 8 types, 64/wave")


@pytest.mark.parametrize("cap", [65535, 70000])
def test_nested_long_output_rows(cap):
    """Output-length rows of 65,534 and 69,999 entries: the largest row the
    kernel's 16-bit search guide covers, and one past it (the guide is then
    off and the whole row is searched).  Short geometric lengths (mean 40)
    with the rest of the row saturated, two segments, every replica against
    the oracle."""
    from tests.gpu_util import check
    B = sim_module()
    rng = np.random.default_rng(cap)
    cdf = np.stack([W.geometric_cdf_table(40.0, cap), W.geometric_cdf_table(25.0, cap)])
    wl = W.Workload(prompt_len=[16, 48], lam=[0.05, 0.03], d0=5.0, d1=0.001, C=cap + 4096,
                    policy="nested", n=[2, 1], out_cap=cap, out_cdf=cdf, seg_end=[64, cap],
                    hist_edges=W.default_edges(5.0, 40), record_capacity=1 << 12)
    check(B, [W.Job(wl, int(rng.integers(0, 2**63)), W.ids(9))], 600,
          f"nested, output rows of {cap - 1} entries")
