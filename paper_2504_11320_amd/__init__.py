"""MI355X-native batched Monte Carlo simulator of the WAIT / Nested WAIT /
FCFS LLM-inference scheduling model (arXiv 2504.11320).

The simulation runs in the HIP library ``libwait_sim.so`` behind the C ABI of
``include/wait_sim.h``; ``binding`` marshals arguments and device buffers.
``calibrate`` (fluid boundary, threshold calibration) and ``analysis``
(metrics, percentiles, the stability point of a rate sweep) are host-side
helpers around it.
"""
from . import analysis, calibrate  # noqa: F401
from .binding import (Simulation, WaitSimError, lib, run_batch,  # noqa: F401
                      split_by_job)

__all__ = ["Simulation", "WaitSimError", "lib", "run_batch", "split_by_job", "analysis",
           "calibrate"]
