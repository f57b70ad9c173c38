// hb_fast_ttg_512s.hip -- instantiations of the fast TreeTraversal kernel with
// leaf records in global memory, for 512-row workgroups with half-size tree chunks.
#include "hb_fast.h"

namespace hb {

FastFn fast_ttg_kernel_512s(int lg, bool multi) {
  return multi ? pick_fast<2, true, 512, kFastTableSmall>(lg) : pick_fast<2, false, 512, kFastTableSmall>(lg);
}

}  // namespace hb
