// sim_known_wait_tv.hip -- instantiates the known-length simulation kernel for
// WAIT (Algorithm 1) for launches with time-varying arrival rates or an
// arrival list.
#include "sim_known_impl.h"

namespace wsim {

hipError_t launch_known_wait_tv(int max_m, const KArgs &A, hipStream_t s) {
  return launch_pol<WS_WAIT, true>(max_m, A, s);
}

}  // namespace wsim
