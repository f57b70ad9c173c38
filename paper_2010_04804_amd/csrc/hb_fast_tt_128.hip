// hb_fast_tt_128.hip -- instantiations of the fast TreeTraversal kernel for
// 128-row workgroups with half-size tree chunks.
#include "hb_fast.h"

namespace hb {

FastFn fast_tt_kernel_128(int lg, int km) {
  return km == 1 ? pick_fast<1, 1, 128, kFastTableSmall>(lg) : pick_fast<1, HB_MAX_OUTPUTS, 128, kFastTableSmall>(lg);
}

}  // namespace hb
