// hb_fast_tt_512s.hip -- instantiations of the fast TreeTraversal kernel for
// 512-row workgroups with half-size tree chunks.
#include "hb_fast.h"

namespace hb {

FastFn fast_tt_kernel_512s(int lg, bool multi) {
  return multi ? pick_fast<1, true, 512, kFastTableSmall>(lg) : pick_fast<1, false, 512, kFastTableSmall>(lg);
}

}  // namespace hb
