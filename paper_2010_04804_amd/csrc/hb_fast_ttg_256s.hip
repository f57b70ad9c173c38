// hb_fast_ttg_256s.hip -- instantiations of the fast TreeTraversal kernel with
// leaf records in global memory, for 256-row workgroups with half-size tree chunks.
#include "hb_fast.h"

namespace hb {

FastFn fast_ttg_kernel_256s(int lg, bool multi) {
  return multi ? pick_fast<2, true, 256, kFastTableSmall>(lg) : pick_fast<2, false, 256, kFastTableSmall>(lg);
}

}  // namespace hb
