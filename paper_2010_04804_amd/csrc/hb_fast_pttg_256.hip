// hb_fast_pttg_256.hip -- instantiations of the fast PerfectTreeTraversal
// kernel with the leaf values in global memory (mode 3) for 256-row
// workgroups: scalar leaves (one output, or one per tree class), depth <= 8, 8-bit leaf-slot ids.
#include "hb_fast.h"

namespace hb {

FastFn fast_pttg_kernel_256(int lg, int km) {
  return km == 1 ? pick_fast<3, 1, 256, kFastTableSmall>(lg)
         : km == 2 ? pick_fast<3, 2, 256, kFastTableSmall>(lg)
                   : pick_fast<3, HB_MAX_OUTPUTS, 256, kFastTableSmall>(lg);
}

}  // namespace hb
