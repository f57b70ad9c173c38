// hb_fast_ttg_256.hip -- instantiations of the fast TreeTraversal kernel with
// leaf records in global memory, for 256-row workgroups.
#include "hb_fast.h"

namespace hb {

FastFn fast_ttg_kernel_256(int lg, bool multi) {
  return multi ? pick_fast<2, true, 256, kFastTableLds>(lg) : pick_fast<2, false, 256, kFastTableLds>(lg);
}

}  // namespace hb
