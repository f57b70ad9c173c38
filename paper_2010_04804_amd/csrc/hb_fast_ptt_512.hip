// hb_fast_ptt_512.hip -- instantiations of the fast PerfectTreeTraversal kernel
// for 512-row workgroups (one translation unit each, so they build in parallel).
#include "hb_fast.h"

namespace hb {

FastFn fast_ptt_kernel_512(int lg, int km) {
  return km == 1 ? pick_fast<0, 1, 512, kFastTableLds>(lg) : pick_fast<0, HB_MAX_OUTPUTS, 512, kFastTableLds>(lg);
}

}  // namespace hb
