// hb_fast_ttg_256.hip -- instantiations of the fast TreeTraversal kernel with
// leaf records in global memory, for 256-row workgroups.
#include "hb_fast.h"

namespace hb {

FastFn fast_ttg_kernel_256(int lg, int km) {
  return km == 1 ? pick_fast<2, 1, 256, kFastTableLds>(lg) : pick_fast<2, HB_MAX_OUTPUTS, 256, kFastTableLds>(lg);
}

}  // namespace hb
