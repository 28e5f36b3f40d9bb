// sim_fcfs_dist.hip -- instantiates the kernel for FCFS with output lengths
// drawn per request (Section 4.1's FCFS under Section 5.1's unknown lengths).
#include "sim_fcfs_dist_impl.h"

namespace wsim {

hipError_t launch_fcfs_dist(int max_m, const KArgs &A, hipStream_t s) {
  // the per-batch trace runs in the general instantiation
  if (A.btrace != nullptr) return launch_fcfs_dist_k<true>(max_m, A, s);
  return launch_fcfs_dist_k<false>(max_m, A, s);
}

}  // namespace wsim
