// hb_fast_tt_1024.hip -- instantiations of the fast TreeTraversal kernel for
// 1024-row workgroups with half-size tree chunks (four waves per SIMD where
// the feature tile is narrow). Single-output only, as for PTT.
#include "hb_fast.h"

namespace hb {

FastFn fast_tt_kernel_1024(int lg, int km) {
  return km == 1 ? pick_fast<1, 1, 1024, kFastTableSmall>(lg) : km == 2 ? pick_fast<1, 2, 1024, kFastTableSmall>(lg) : nullptr;
}

}  // namespace hb
