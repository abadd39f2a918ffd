// fold_part.hip -- the folded kernels (three planes, and one plane for
// fixed-point scales) writing the raw integer sums of one K split each.
#include "fold_kernel.h"

namespace fgq {

fgq_status launch_fold_part(const FoldArgs& a, int bits, hipStream_t st) { return launch_out<1, false>(a, bits, st); }

fgq_status launch_fold_dfp_part(const FoldArgs& a, int bits, hipStream_t st) {
  return launch_out<1, true>(a, bits, st);
}

}  // namespace fgq
