// hb_fast_ptt_768.hip -- instantiations of the fast PerfectTreeTraversal kernel
// for 768-row workgroups with half-size tree chunks (three waves per SIMD).
#include "hb_fast.h"

namespace hb {

// Single-output only: the multi-output accumulators do not fit in the
// registers three waves per SIMD leave.
FastFn fast_ptt_kernel_768(int lg, int km) {
  return km == 1 ? pick_fast<0, 1, 768, kFastTableSmall>(lg) : km == 2 ? pick_fast<0, 2, 768, kFastTableSmall>(lg) : nullptr;
}

}  // namespace hb
