// hb_fast_ptt_128.hip -- instantiations of the fast PerfectTreeTraversal kernel
// for 128-row workgroups with half-size tree chunks: rows of a few hundred
// features whose tile would not fit at 256 rows.
#include "hb_fast.h"

namespace hb {

FastFn fast_ptt_kernel_128(int lg, int km) {
  return km == 1 ? pick_fast<0, 1, 128, kFastTableSmall>(lg) : pick_fast<0, HB_MAX_OUTPUTS, 128, kFastTableSmall>(lg);
}

}  // namespace hb
