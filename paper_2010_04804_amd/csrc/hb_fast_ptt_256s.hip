// hb_fast_ptt_256s.hip -- instantiations of the fast PerfectTreeTraversal kernel
// for 256-row workgroups with half-size tree chunks (feature tiles of about
// a hundred columns, which leave no room for a full chunk at 256 rows).
#include "hb_fast.h"

namespace hb {

FastFn fast_ptt_kernel_256s(int lg, int km) {
  return km == 1 ? pick_fast<0, 1, 256, kFastTableSmall>(lg) : pick_fast<0, HB_MAX_OUTPUTS, 256, kFastTableSmall>(lg);
}

}  // namespace hb
