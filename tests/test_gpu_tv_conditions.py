"""The time-varying threshold conditions on the GPU (the appendix on
time-varying arrival rates: the window load Lambda^pi over a full batch's
service time must stay below n_1, and the worst continuation probabilities
below n_k / n_{k-1}).  Nested WAIT with thresholds (6, 3, 1) under intensity
lam (1 + 0.3 sin(2 pi t / 6000 ms)): at lam = 2.9 the host calculator finds
Lambda^pi = 5.68 < 6 and the entry queue stays short; at lam = 3.4 (average
load still below 6 per batch) Lambda^pi = 6.65 > 6 and the queue builds up
during every peak.  Per-batch traces of 512 replicas x 12,000 batches; two
replicas' traces equal the oracle's batch by batch."""
import numpy as np
import pytest

import workloads as W
from paper_2504_11320_amd import calibrate as K
from tests.gpu_util import sim_module

pytestmark = pytest.mark.gpu


def _model(lam):
    probs = {8: 0.6, 24: 0.3, 64: 0.1}
    F, acc = [], 0.0
    for s in range(1, 64):
        acc += probs.get(s, 0.0)
        F.append(acc)
    row = W._cdf_table(F)
    rt = np.linspace(0.0, 2.4e4, 32)
    f = 1.0 + 0.3 * np.sin(2.0 * np.pi * rt / 6000.0)
    wl = W.Workload(prompt_len=[16], lam=[lam], d0=1.0, d1=1e-4, C=100000, policy="nested",
                    n=[6, 3, 1], out_cap=64, out_cdf=row[None, :], seg_end=[8, 24, 64],
                    hist_edges=W.default_edges(1.0, 32), record_capacity=1 << 16,
                    rate_t=rt, rate_f=f[None, :])
    return wl, row


def test_window_load_condition_predicts_queue_growth():
    B = sim_module()
    from oracle import oracle as O
    H, R = 12000, 512
    peak = {}
    for lam in (2.9, 3.4):
        wl, row = _model(lam)
        delta = wl.d0 + wl.d1 * K.base_memory(wl.n, wl.seg_end, 16)   # full batch
        seg = K.segment_intensities(wl.lam, wl.rate_t, wl.rate_f, wl.seg_end,
                                    cdf=row[None, :], cap=64)
        chk = K.check_time_varying(wl.lam, wl.rate_t, wl.rate_f, wl.n, delta, 2.4e4,
                                   seg_inten=seg)
        assert chk["continuation_ok"]
        assert chk["load_ok"] == (lam == 2.9), chk["Lambda_pi"]
        sim = B.Simulation([W.Job(wl, 0, W.ids(R))])
        sim.prepare()
        print(f"[gpu] time-varying conditions: lam {lam}, Lambda_pi "
              f"{chk['Lambda_pi']:.3f}, {R} replicas x {H}", flush=True)
        tr = sim.advance_traced(H, H)
        res = sim.results()
        assert np.all(res["batches"] == H)
        peak[lam] = float(tr["waiting_after"].max(axis=1).mean())
        for x in (0, R - 1):
            o = O.run_one(wl, 0, x, H, btrace_cap=H)
            for b in range(0, H, 997):
                rec = o["batches_trace"][b]
                for fld in ("tokens", "selected", "completions", "waiting_after",
                            "resident_after", "mem_after"):
                    assert tr[x][b][fld] == rec[fld], (lam, x, b, fld)
    print(f"[gpu] time-varying conditions: mean peak entry queue {peak}", flush=True)
    assert peak[2.9] < 50 and peak[3.4] > 80
