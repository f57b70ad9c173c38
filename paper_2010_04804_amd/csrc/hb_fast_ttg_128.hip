// hb_fast_ttg_128.hip -- instantiations of the fast TreeTraversal kernel with
// leaf records in global memory, for 128-row workgroups with half-size tree
// chunks.
#include "hb_fast.h"

namespace hb {

FastFn fast_ttg_kernel_128(int lg, int km) {
  return km == 1 ? pick_fast<2, 1, 128, kFastTableSmall>(lg) : pick_fast<2, HB_MAX_OUTPUTS, 128, kFastTableSmall>(lg);
}

}  // namespace hb
