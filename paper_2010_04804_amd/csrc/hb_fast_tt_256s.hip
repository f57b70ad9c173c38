// hb_fast_tt_256s.hip -- instantiations of the fast TreeTraversal kernel for
// 256-row workgroups with half-size tree chunks.
#include "hb_fast.h"

namespace hb {

FastFn fast_tt_kernel_256s(int lg, bool multi) {
  return multi ? pick_fast<1, true, 256, kFastTableSmall>(lg) : pick_fast<1, false, 256, kFastTableSmall>(lg);
}

}  // namespace hb
