// sim_known_wait.hip -- instantiates the known-length simulation kernel for
// WAIT (Algorithm 1) with constant arrival rates.
#include "sim_known_impl.h"

namespace wsim {

hipError_t launch_known_wait(int max_m, const KArgs &A, hipStream_t s) {
  if (A.any_trace || A.any_tv || A.btrace != nullptr) return launch_known_wait_tv(max_m, A, s);
  return launch_pol<WS_WAIT, false>(max_m, A, s);
}

}  // namespace wsim
