"""The eviction-probability guarantee of Nested WAIT's segment design on the
GPU (the theorem on Nested WAIT with L segments, memory condition
C >= M_req): thresholds meeting the drift conditions, C from the host
calculator's M_req for delta = 0.05, 8192 replicas x 10^5 batches.  The
fraction of replicas with any eviction is at most delta; with the
deterministic part of the bound only (M^pi plus the boundary term, no
logarithmic buffer) most replicas evict.  Sampled replicas equal the
oracle's."""
import math

import numpy as np
import pytest

import workloads as W
from paper_2504_11320_amd import calibrate as K
from tests.gpu_util import sim_module
from tests.parity_util import compare

pytestmark = pytest.mark.gpu


def _model(C):
    # common prompt 16; outputs 8 / 24 / 64 with probabilities 0.6 / 0.3 / 0.1
    probs = {8: 0.6, 24: 0.3, 64: 0.1}
    F, acc = [], 0.0
    for s in range(1, 64):
        acc += probs.get(s, 0.0)
        F.append(acc)
    row = W._cdf_table(F)
    return W.Workload(prompt_len=[16], lam=[3.5], d0=1.0, d1=1e-4, C=C, policy="nested",
                      n=[6, 3, 1], out_cap=64, out_cdf=row[None, :], seg_end=[8, 24, 64],
                      hist_edges=W.default_edges(1.0, 32), record_capacity=1 << 16), row


def test_eviction_probability_at_m_req():
    B = sim_module()
    from oracle import oracle as O
    H, delta = 100000, 0.05
    wl0, row = _model(10**6)
    seg_rates = K.segment_rates(wl0.lam, wl0.seg_end, cdf=row[None, :], cap=64)
    p = K.continuation_probabilities(seg_rates)
    n = wl0.n
    # the drift conditions: Delta T(n) < n_1 / Lambda, p_k < n_k / n_{k-1} < 1
    assert wl0.d0 + wl0.d1 * K.base_memory(n, wl0.seg_end, 16) < n[0] / sum(seg_rates)
    assert all(p[k - 1] < n[k] / n[k - 1] < 1 for k in (1, 2))
    # processing opportunities over the horizon: at most H batches, each >= d0
    zT = 2.0 * H * (wl0.d0 + wl0.d1 * K.base_memory(n, wl0.seg_end, 16))
    req = K.memory_requirement(n, wl0.seg_end, 16, p, 3, zT, wl0.d0, delta)
    reps = W.ids(8192)
    fr = {}
    for name, C in (("M_req", math.ceil(req["total"])),
                    ("M_pi + boundary", math.ceil(req["term1"] + req["term2"]))):
        wl, _ = _model(int(C))
        print(f"[gpu] memory bound: C = {C} ({name}), {len(reps)} replicas x {H}", flush=True)
        g = B.run_batch([W.Job(wl, 3, reps)], H)
        assert np.all(g["batches"] == H) and np.all(g["t_end"] <= zT)
        fr[name] = float(np.mean(g["evictions"] > 0))
        sub = W.Job(wl, 3, reps[[0, 8191]])
        o = O.run_job(sub, H)
        compare({k: v[[0, 8191]] for k, v in g.items()}, o, f"memory bound {name}")
    print(f"[gpu] memory bound: fraction of replicas with an eviction: {fr}", flush=True)
    assert fr["M_req"] <= delta
    assert fr["M_pi + boundary"] > 0.5
