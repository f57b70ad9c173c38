// hb_fast_tt_128.hip -- instantiations of the fast TreeTraversal kernel for
// 128-row workgroups with half-size tree chunks.
#include "hb_fast.h"

namespace hb {

FastFn fast_tt_kernel_128(int lg, bool multi) {
  return multi ? pick_fast<1, true, 128, kFastTableSmall>(lg) : pick_fast<1, false, 128, kFastTableSmall>(lg);
}

}  // namespace hb
