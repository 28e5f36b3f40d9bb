// sim_wait_many.hip -- instantiates the WAIT kernel for more than 16 request
// types (Algorithm 1 with per-type state in LDS columns).
#include "sim_wait_many_impl.h"

namespace wsim {

hipError_t launch_wait_many(int max_m, const KArgs &A, hipStream_t s) {
  // arrival lists and per-batch traces run in the general instantiation
  if (A.any_trace || A.btrace != nullptr) return launch_wait_many_k<true>(max_m, A, s);
  return launch_wait_many_k<false>(max_m, A, s);
}

}  // namespace wsim
