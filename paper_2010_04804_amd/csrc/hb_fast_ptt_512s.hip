// hb_fast_ptt_512s.hip -- instantiations of the fast PerfectTreeTraversal kernel
// for 512-row workgroups with half-size tree chunks (for feature tiles too
// wide to sit beside a full chunk: eight waves per CU instead of four).
#include "hb_fast.h"

namespace hb {

FastFn fast_ptt_kernel_512s(int lg, int km) {
  return km == 1 ? pick_fast<0, 1, 512, kFastTableSmall>(lg) : pick_fast<0, HB_MAX_OUTPUTS, 512, kFastTableSmall>(lg);
}

}  // namespace hb
