// hb_fast_tt_512.hip -- instantiations of the fast TreeTraversal kernel
// for 512-row workgroups (one translation unit each, so they build in parallel).
#include "hb_fast.h"

namespace hb {

FastFn fast_tt_kernel_512(int lg, int km) {
  return km == 1 ? pick_fast<1, 1, 512, kFastTableLds>(lg) : pick_fast<1, HB_MAX_OUTPUTS, 512, kFastTableLds>(lg);
}

}  // namespace hb
