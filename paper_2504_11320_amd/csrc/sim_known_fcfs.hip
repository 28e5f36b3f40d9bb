// sim_known_fcfs.hip -- instantiates the known-length simulation kernel for
// greedy FCFS with LIFO eviction on overflow (Section 4.1) with constant
// arrival rates.
#include "sim_known_impl.h"

namespace wsim {

hipError_t launch_known_fcfs(int max_m, const KArgs &A, hipStream_t s) {
  if (A.any_trace || A.any_tv || A.btrace != nullptr) return launch_known_fcfs_tv(max_m, A, s);
  return launch_pol<WS_FCFS, false>(max_m, A, s);
}

}  // namespace wsim
