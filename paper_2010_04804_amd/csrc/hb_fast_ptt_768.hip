// hb_fast_ptt_768.hip -- instantiations of the fast PerfectTreeTraversal kernel
// for 768-row workgroups with half-size tree chunks (three waves per SIMD).
#include "hb_fast.h"

namespace hb {

// Single-output only: the multi-output accumulators do not fit in the
// registers three waves per SIMD leave.
FastFn fast_ptt_kernel_768(int lg, bool multi) {
  return multi ? nullptr : pick_fast<0, false, 768, kFastTableSmall>(lg);
}

}  // namespace hb
