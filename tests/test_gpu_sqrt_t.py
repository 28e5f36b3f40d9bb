"""The square-root law at the boundary on the GPU (the proposition on the
sqrt(T) lower bound, Section 4.3): single-type WAIT at critical load
(lambda Delta T = n) over 8192 replicas and horizons 10^3 to 2.56 x 10^5
batches.  The mean censored latency grows like the square root of the horizon
(x256 in horizon, about x16 in latency), a subcritical load keeps it flat, and
sampled replicas equal the oracle's."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import sim_module
from tests.parity_util import compare
from tests.test_review_and_sqrt_t import _critical

pytestmark = pytest.mark.gpu


def test_sqrt_t_on_gpu():
    B = sim_module()
    from oracle import oracle as O
    reps = W.ids(8192)
    lat = {}
    for lam in (2.0, 1.6):
        for H in (1000, 16000, 256000):
            print(f"[gpu] sqrt-T: lam {lam}, horizon {H}", flush=True)
            g = B.run_batch([W.Job(_critical(lam), 7, reps)], H)
            assert np.all(g["flags"] == 0) and np.all(g["batches"] == H)
            lat[lam, H] = float((g["lat_area"] / g["arrivals"]).mean())
            if H == 16000:
                sub = W.Job(_critical(lam), 7, reps[[0, 4095, 8191]])
                o = O.run_job(sub, H)
                gs = {k: v[[0, 4095, 8191]] for k, v in g.items()}
                compare(gs, o, f"sqrt-T lam {lam}")
    crit = lat[2.0, 256000] / lat[2.0, 1000]
    flat = lat[1.6, 256000] / lat[1.6, 1000]
    print(f"[gpu] sqrt-T: latency ratio x256 horizon: critical {crit:.2f}, "
          f"subcritical {flat:.3f}", flush=True)
    assert 11.0 < crit < 19.0
    assert 0.9 < flat < 1.1
