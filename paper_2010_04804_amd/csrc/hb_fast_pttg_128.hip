// hb_fast_pttg_128.hip -- instantiations of the fast PerfectTreeTraversal
// kernel with the leaf values in global memory (mode 3) for 128-row
// workgroups: one output, depth <= 8, 8-bit leaf-slot ids.
#include "hb_fast.h"

namespace hb {

FastFn fast_pttg_kernel_128(int lg, int km) { return km == 1 ? pick_fast<3, 1, 128, kFastTableSmall>(lg) : nullptr; }

}  // namespace hb
