// hb_fast_ptt_1024.hip -- instantiations of the fast PerfectTreeTraversal
// kernel for 1024-row workgroups with half-size tree chunks (four waves per
// SIMD where the feature tile is narrow). Single-output only: the
// multi-output accumulators do not fit in the registers four waves leave.
#include "hb_fast.h"

namespace hb {

FastFn fast_ptt_kernel_1024(int lg, int km) {
  return km == 1 ? pick_fast<0, 1, 1024, kFastTableSmall>(lg) : km == 2 ? pick_fast<0, 2, 1024, kFastTableSmall>(lg) : nullptr;
}

}  // namespace hb
