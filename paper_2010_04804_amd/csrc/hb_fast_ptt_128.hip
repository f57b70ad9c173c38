// hb_fast_ptt_128.hip -- instantiations of the fast PerfectTreeTraversal kernel
// for 128-row workgroups with half-size tree chunks: rows of a few hundred
// features whose tile would not fit at 256 rows.
#include "hb_fast.h"

namespace hb {

FastFn fast_ptt_kernel_128(int lg, bool multi) {
  return multi ? pick_fast<0, true, 128, kFastTableSmall>(lg) : pick_fast<0, false, 128, kFastTableSmall>(lg);
}

}  // namespace hb
