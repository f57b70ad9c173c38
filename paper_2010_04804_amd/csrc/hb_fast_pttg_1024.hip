// hb_fast_pttg_1024.hip -- instantiations of the fast PerfectTreeTraversal
// kernel with the leaf values in global memory (mode 3) for 1024-row
// workgroups: scalar leaves (one output, or one per tree class), depth <= 8, 8-bit leaf-slot ids.
#include "hb_fast.h"

namespace hb {

FastFn fast_pttg_kernel_1024(int lg, int km) {
  // sixteen double accumulators do not fit in the registers four waves per SIMD leave
  return km == 1 ? pick_fast<3, 1, 1024, kFastTableSmall>(lg) : km == 2 ? pick_fast<3, 2, 1024, kFastTableSmall>(lg) : nullptr;
}

}  // namespace hb
