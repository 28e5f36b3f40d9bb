"""GPU parity of Nested WAIT (Algorithm 2 / Algorithm 4) against the oracle."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import check, sim_module

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    return sim_module()


def test_nested_traces(B):
    d1 = 0.01
    d0 = 1.0 - 12 * d1
    times = [1e-4 * i for i in range(200)]
    # full prefix batch = M^pi, no eviction
    wl = W.trace_workload("nested", [1], None, d0, d1, 40, [4, 2], times, [0] * 200,
                          lengths=[1 + (i % 2) for i in range(200)], seg_end=[1, 2],
                          out_cap=2)
    g, _ = check(B, [W.Job(wl, 0, W.ids(2))], 12, "nested trace M^pi")
    assert g["evictions"][0] == 0
    # boundary-only repair when C >= M^pi
    wl = W.trace_workload("nested", [10], None, 1.0, 0.001, 200, [2, 1], times[:400],
                          [0] * 200, lengths=[8] * 200, seg_end=[2, 8], out_cap=8)
    g, _ = check(B, [W.Job(wl, 0, W.ids(2))], 80, "nested trace boundary repair")
    assert g["evictions"][0] > 0 and g["fallback_evictions"][0] == 0
    # below M^pi: interior fallback
    wl = W.trace_workload("nested", [10], None, 1.0, 0.001, 150, [4, 1], times, [0] * 200,
                          lengths=[8] * 200, seg_end=[2, 8], out_cap=8)
    g, _ = check(B, [W.Job(wl, 0, W.ids(2))], 60, "nested trace fallback")
    assert g["fallback_evictions"][0] > 0


def test_config3_subset(B):
    jobs = W.config3(replicas=70, rate_index=[0, 16, 31])
    check(B, jobs, 3000, "config3 3 rates x70 x3000")


def test_config5_subset(B):
    jobs = W.config5(replicas=96)
    check(B, jobs, 1500, "config5 96 x1500")


def test_nested_resume(B):
    jobs = W.config3(replicas=64, rate_index=[3, 29])
    one = B.run_batch(jobs, 2000)
    s = B.Simulation(jobs)
    s.prepare()
    s.advance(700, resume=False)
    s.advance(1300, resume=True)
    two = s.results()
    for k in one:
        assert np.array_equal(one[k], two[k]), k


def test_nested_known_lengths_and_thin_segments(B):
    # known lengths under Nested WAIT, a width-1 segment and a single segment
    wl = W.Workload(prompt_len=[8, 20], lam=[0.3, 0.2], d0=2.0, d1=0.01, C=600,
                    policy="nested", n=[3, 2, 1], out_len=[4, 9], seg_end=[4, 5, 9],
                    hist_edges=W.default_edges(2.0, 80))
    check(B, [W.Job(wl, 5, W.ids(67))], 1500, "nested known lengths, width-1 segment")
    wl1 = W.Workload(prompt_len=[8, 20], lam=[0.3, 0.2], d0=2.0, d1=0.01, C=400,
                     policy="nested", n=[2], out_cap=12,
                     out_cdf=np.stack([W.geometric_cdf_table(3.0, 12)] * 2),
                     seg_end=[12], hist_edges=W.default_edges(2.0, 80))
    check(B, [W.Job(wl1, 9, W.ids(40))], 1500, "nested single segment")
