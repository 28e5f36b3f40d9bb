// sim_known_wait.hip -- instantiates the known-length simulation kernel for
// WAIT (Algorithm 1).
#include "sim_known_impl.h"

namespace wsim {

hipError_t launch_known_wait(int max_m, const KArgs &A, hipStream_t s) {
  return launch_pol<WS_WAIT>(max_m, A, s);
}

}  // namespace wsim
