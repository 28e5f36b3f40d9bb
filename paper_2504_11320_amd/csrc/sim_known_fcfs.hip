// sim_known_fcfs.hip -- instantiates the known-length simulation kernel for
// greedy FCFS with LIFO eviction on overflow (Section 4.1).
#include "sim_known_impl.h"

namespace wsim {

hipError_t launch_known_fcfs(int max_m, const KArgs &A, hipStream_t s) {
  return launch_pol<WS_FCFS>(max_m, A, s);
}

}  // namespace wsim
