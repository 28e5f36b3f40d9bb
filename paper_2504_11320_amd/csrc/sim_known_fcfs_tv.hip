// sim_known_fcfs_tv.hip -- instantiates the known-length simulation kernel
// for greedy FCFS (Section 4.1) for launches with time-varying arrival rates
// or an arrival list.
#include "sim_known_impl.h"

namespace wsim {

hipError_t launch_known_fcfs_tv(int max_m, const KArgs &A, hipStream_t s) {
  return launch_pol<WS_FCFS, true>(max_m, A, s);
}

}  // namespace wsim
