"""GPU parity with time-varying arrival rates (the paper's appendix on
time-varying rates: type j arrives at lam_j f_j(t), sampled by thinning).
Every test compares the HIP library element by element with the oracle on the
same seeded streams, or one launch layout with another."""
import math

import numpy as np
import pytest

import workloads as W
from tests.gpu_util import check, sim_module

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    return sim_module()


def _profile(rng, m, span, P=None):
    """Random profile: P points over [0, span], factors in [0, 2] with some
    exact zeros (zero stretches), per type."""
    P = P or int(rng.integers(1, 12))
    t = np.sort(rng.uniform(0.0, span, P))
    t = np.unique(t)
    f = rng.uniform(0.0, 2.0, (m, len(t)))
    f[rng.uniform(size=f.shape) < 0.2] = 0.0
    return t, f


def _llama(policy, rate_index=16):
    wl = W.config2(replicas=1, rate_index=[rate_index])[0].wl
    wl.policy = policy
    wl.n = [] if policy == "fcfs" else [2, 1, 1]
    return wl


def test_every_policy_with_a_profile(B):
    """WAIT, WAIT-no-wait, FCFS and Nested WAIT (known and unknown lengths)
    under the cyclic profile, with a constant-rate job in the same launches."""
    span = 3.0e6
    rt, rf = W.diurnal_profile(3, span, points=13, cycles=2.0)
    jobs = []
    for pol in ("wait", "wait-nowait", "fcfs"):
        wl = W.with_profile(_llama(pol), rt, rf)
        jobs.append(W.Job(wl, 5, W.ids(37)))
    jobs.append(W.Job(_llama("wait"), 5, W.ids(11)))  # constant rates, same launch
    nest = W.config3(replicas=1, rate_index=[20])[0].wl
    jobs.append(W.Job(W.with_profile(nest, rt, rf), 6, W.ids(29)))
    nk = W.Workload(prompt_len=[16, 64, 128], lam=[0.02, 0.01, 0.005], d0=5.0, d1=0.01,
                    C=3000, policy="nested", n=[2, 1, 1], out_len=[8, 20, 40],
                    seg_end=[8, 20, 40], hist_edges=W.default_edges(5.0, 100))
    rt2, rf2 = W.diurnal_profile(3, 2.0e4, points=9, amp=0.9)
    jobs.append(W.Job(W.with_profile(nk, rt2, rf2), 7, W.ids(23)))
    g, o = check(B, jobs, 1500, "time-varying rates, 4 policies")
    assert g["arrivals"].min() > 0


def test_zero_stretches_and_stop(B):
    """Profiles with zero stretches and an intensity that ends at zero: no
    arrivals there, replicas stall once every type has stopped."""
    rt = np.array([0.0, 5.0e4, 1.0e5, 2.0e5, 2.5e5, 3.0e5])
    rf = np.array([[0.0, 1.0, 0.0, 0.0, 2.0, 0.0],
                   [1.0, 1.0, 0.0, 0.0, 1.0, 0.0],
                   [0.5, 0.0, 0.0, 3.0, 0.0, 0.0]])
    wls = [W.with_profile(_llama(p), rt, rf) for p in ("wait", "fcfs")]
    nest = W.with_profile(W.config3(replicas=1, rate_index=[31])[0].wl, rt, rf)
    jobs = [W.Job(wls[0], 3, W.ids(19)), W.Job(wls[1], 3, W.ids(19)), W.Job(nest, 3, W.ids(19))]
    g, o = check(B, jobs, 4000, "zero stretches, intensities ending at zero")
    assert np.all(g["flags"] & 2)  # every replica stalled once arrivals ended


def test_constant_profile_equals_constant_rates(B):
    """A constant profile f_j = c_j on the GPU reproduces the constant-rate
    run at lam_j c_j bit for bit."""
    c = np.array([1.5, 0.5, 1.0])
    base = _llama("wait")
    tv = W.with_profile(base, [0.0, 1.0e6], np.stack([c, c], axis=1))
    hom = W.Workload(**{**base.__dict__, "lam": [x * y for x, y in zip(base.lam, c)]})
    a = B.run_batch([W.Job(tv, 9, W.ids(40))], 2000)
    b = B.run_batch([W.Job(hom, 9, W.ids(40))], 2000)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_random_profiles(B):
    """Seeded random small models and random profiles over every policy."""
    from tests.test_gpu_random import random_workload
    rng = np.random.default_rng(77)
    jobs = []
    for i in range(24):
        wl = random_workload(rng)
        rt, rf = _profile(rng, wl.m, float(rng.uniform(50.0, 5000.0)))
        jobs.append(W.Job(W.with_profile(wl, rt, rf), int(rng.integers(0, 2**63)),
                          W.ids(int(rng.integers(1, 50)))))
    check(B, jobs, 600, "24 random models with random profiles")


def test_trace_and_profile_in_one_launch(B):
    """A replayed arrival list and a profiled job share the WAIT launch."""
    tr = W.trace_workload("wait", [16, 32], [4, 8], 5.0, 0.01, 1000, [2, 1],
                          [0.0, 0.0, 1.0, 2.5, 9.0, 9.0, 30.0], [0, 1, 0, 0, 1, 1, 0])
    rt, rf = W.diurnal_profile(3, 5.0e5, points=7)
    jobs = [W.Job(tr, 1, W.ids(3)), W.Job(W.with_profile(_llama("wait"), rt, rf), 2, W.ids(21))]
    check(B, jobs, 800, "arrival list and profile, one launch")


def test_resume_matches_one_call(B):
    """Two advances of h/2 batches equal one of h."""
    rt, rf = W.diurnal_profile(3, 2.0e6, points=11)
    jobs = [W.Job(W.with_profile(_llama("wait"), rt, rf), 4, W.ids(33)),
            W.Job(W.with_profile(W.config3(replicas=1, rate_index=[10])[0].wl, rt, rf), 4,
                  W.ids(17))]
    one = B.run_batch(jobs, 1200)
    sim = B.Simulation(jobs)
    sim.prepare()
    sim.advance(600, resume=False)
    sim.advance(600, resume=True)
    two = sim.results()
    for k in one:
        assert np.array_equal(one[k], two[k]), k


def test_thinning_limit_flag(B):
    """A positive intensity 2^-30 of its bound: the GPU flags the rejection
    limit exactly where the oracle does."""
    wl = W.Workload(prompt_len=[16], lam=[1.0], d0=5.0, d1=0.01, C=1000, policy="wait",
                    n=[1], out_len=[4], hist_edges=W.default_edges(5.0, 16),
                    rate_t=np.array([0.0, 1.0]), rate_f=np.array([[1.0, 2.0 ** -30]]))
    g, o = check(B, [W.Job(wl, 4, W.ids(2))], 50, "thinning rejection limit")
    assert np.all(g["flags"] & 8)


def test_random_profiles_with_chunked_fcfs(B):
    """Random profiles combined with chunked-prefill FCFS (budgets 5-200
    tokens) and with the other policies, in one launch per policy."""
    from tests.test_gpu_random import random_workload
    rng = np.random.default_rng(78)
    jobs = []
    while len(jobs) < 20:
        wl = random_workload(rng)
        if wl.policy == "fcfs":
            wl.chunk = int(rng.integers(5, 200))
        elif len(jobs) % 3:
            continue
        rt, rf = _profile(rng, wl.m, float(rng.uniform(50.0, 5000.0)))
        jobs.append(W.Job(W.with_profile(wl, rt, rf), int(rng.integers(0, 2**63)),
                          W.ids(int(rng.integers(1, 40)))))
    check(B, jobs, 600, "random profiles with chunked FCFS")
