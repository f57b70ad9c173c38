// hb_fast_ttg_1024.hip -- instantiations of the fast TreeTraversal kernel with
// leaf records in global memory, for 1024-row workgroups with half-size tree
// chunks. Single-output only, as for PTT.
#include "hb_fast.h"

namespace hb {

FastFn fast_ttg_kernel_1024(int lg, int km) {
  return km == 1 ? pick_fast<2, 1, 1024, kFastTableSmall>(lg) : km == 2 ? pick_fast<2, 2, 1024, kFastTableSmall>(lg) : nullptr;
}

}  // namespace hb
