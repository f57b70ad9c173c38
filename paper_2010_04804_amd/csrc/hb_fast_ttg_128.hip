// hb_fast_ttg_128.hip -- instantiations of the fast TreeTraversal kernel with
// leaf records in global memory, for 128-row workgroups with half-size tree
// chunks.
#include "hb_fast.h"

namespace hb {

FastFn fast_ttg_kernel_128(int lg, bool multi) {
  return multi ? pick_fast<2, true, 128, kFastTableSmall>(lg) : pick_fast<2, false, 128, kFastTableSmall>(lg);
}

}  // namespace hb
