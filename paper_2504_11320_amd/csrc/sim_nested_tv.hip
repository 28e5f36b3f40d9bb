// sim_nested_tv.hip -- instantiates the Nested WAIT simulation kernel
// (Algorithm 2) for launches with time-varying arrival rates.
#include "sim_nested_impl.h"

namespace wsim {

hipError_t launch_nested_tv(int max_m, int max_seg, const KArgs &A, hipStream_t s) {
  return launch_nested_k<true>(max_m, max_seg, A, s);
}

}  // namespace wsim
