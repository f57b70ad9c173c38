// hb_fast_tt_512s.hip -- instantiations of the fast TreeTraversal kernel for
// 512-row workgroups with half-size tree chunks.
#include "hb_fast.h"

namespace hb {

FastFn fast_tt_kernel_512s(int lg, int km) {
  return km == 1 ? pick_fast<1, 1, 512, kFastTableSmall>(lg) : pick_fast<1, HB_MAX_OUTPUTS, 512, kFastTableSmall>(lg);
}

}  // namespace hb
