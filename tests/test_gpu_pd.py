"""GPU parity on the decode-only (PD-disaggregated) p630d20 workload: WAIT
with the fluid thresholds and FCFS with a 1 % reserve at 9 rates, against the
oracle."""
import pytest

import workloads as W
from tests.gpu_util import check, sim_module

pytestmark = pytest.mark.gpu


def test_pd_decode_parity():
    B = sim_module()
    jobs = W.config_pd(replicas=21)
    check(B, jobs, 3000, "decode-only p630d20, WAIT and FCFS, 9 rates x21 x3000")
