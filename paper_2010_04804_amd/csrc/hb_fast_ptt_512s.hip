// hb_fast_ptt_512s.hip -- instantiations of the fast PerfectTreeTraversal kernel
// for 512-row workgroups with half-size tree chunks (for feature tiles too
// wide to sit beside a full chunk: eight waves per CU instead of four).
#include "hb_fast.h"

namespace hb {

FastFn fast_ptt_kernel_512s(int lg, bool multi) {
  return multi ? pick_fast<0, true, 512, kFastTableSmall>(lg) : pick_fast<0, false, 512, kFastTableSmall>(lg);
}

}  // namespace hb
