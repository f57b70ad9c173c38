// hb_fast_ptt_768.hip -- instantiations of the fast PerfectTreeTraversal kernel
// for 768-row workgroups with half-size tree chunks (three waves per SIMD).
#include "hb_fast.h"

namespace hb {

FastFn fast_ptt_kernel_768(int lg, bool multi) {
  return multi ? pick_fast<0, true, 768, kFastTableSmall>(lg) : pick_fast<0, false, 768, kFastTableSmall>(lg);
}

}  // namespace hb
