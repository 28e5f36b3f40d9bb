// sim_known_wait.hip -- instantiates the known-length simulation kernel for
// WAIT (Algorithm 1) with constant arrival rates.
#include "sim_known_impl.h"

namespace wsim {

hipError_t launch_known_wait(int max_m, const KArgs &A, hipStream_t s) {
  // more types than the register-resident per-type state holds
  if (max_m > WS_MAX_TYPES_KNOWN) return launch_wait_many(max_m, A, s);
  // arrival lists, time-varying rates, per-batch traces and per-stage caps
  // run in the general instantiation
  if (A.any_trace || A.any_tv || A.btrace != nullptr || A.any_caps)
    return launch_known_wait_tv(max_m, A, s);
  return launch_pol<WS_WAIT, false>(max_m, A, s);
}

}  // namespace wsim
