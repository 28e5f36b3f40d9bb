// sim_nested.hip -- instantiates the Nested WAIT simulation kernel (Algorithm
// 2) for launches with constant arrival rates.
#include "sim_nested_impl.h"

namespace wsim {

hipError_t launch_nested(int max_m, int max_seg, const KArgs &A, hipStream_t s) {
  // time-varying rates, per-batch traces and per-stage caps run in the
  // general instantiation
  if (A.any_tv || A.btrace != nullptr || A.any_caps) return launch_nested_tv(max_m, max_seg, A, s);
  return launch_nested_k<false>(max_m, max_seg, A, s);
}

}  // namespace wsim
