"""wait_sim_run_static (the entry point for callers that cannot allocate
device memory) against wait_sim_run on the same inputs: every result field
equal, on two calls in a row, the second with fewer replicas and a shorter
horizon (so it must not see the first call's state), for WAIT, Nested WAIT
and FCFS; and a job beyond the static workspace is refused with
WS_EWORKSPACE."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import sim_module

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    return sim_module()


def _same(a, b, ctx):
    for k in a:
        if a[k].dtype.kind == "f":
            rel = np.abs(a[k] - b[k]) / np.maximum(np.abs(b[k]), 1e-300)
            assert rel.max(initial=0.0) <= 1e-12, (ctx, k)
        else:
            assert np.array_equal(a[k], b[k]), (ctx, k)


def _jobs():
    wait = W.config2(replicas=48, rate_index=[20])[0]
    nested = W.config3(replicas=40, rate_index=[25])[0]
    nested.wl.record_capacity = 1 << 10
    fcfs = W.config_pd(replicas=32)[-1]
    return [(wait, 1200, 20, 700), (nested, 1500, 9, 400), (fcfs, 900, 17, 300)]


def test_static_entry_matches_run(B):
    for job, h1, n2, h2 in _jobs():
        ja = B.JobArray([job])
        assert B.workspace_bytes(ja) <= B.WS_STATIC_WORKSPACE_BYTES, job.wl.policy
        small = W.Job(job.wl, job.seed, job.replica_ids[:n2])
        print(f"[gpu] run_static {job.wl.policy}: {job.n} x {h1}, then {n2} x {h2}", flush=True)
        got1 = B.run_static(job, h1)
        got2 = B.run_static(small, h2)
        want1 = B.run_batch([job], h1)
        want2 = B.run_batch([small], h2)
        _same(got1, want1, (job.wl.policy, "first"))
        _same(got2, want2, (job.wl.policy, "second"))
        assert got1["batches"].min() > 0


def test_static_entry_refuses_large_jobs(B):
    big = W.config2(replicas=1024, rate_index=[3])[0]
    assert B.workspace_bytes(B.JobArray([big])) > B.WS_STATIC_WORKSPACE_BYTES
    with pytest.raises(B.WaitSimError) as e:
        B.run_static(big, 10)
    assert e.value.code == B.WS_EWORKSPACE
    assert "static workspace" in str(e.value)
