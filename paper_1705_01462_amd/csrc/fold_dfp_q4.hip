// fold_dfp_q4.hip -- the fixed-point-scale layer kernels that emit 4-bit
// codes of the next layer's activations.
#include "fold_kernel.h"

namespace fgq {

fgq_status launch_fold_dfp_out_q4(const FoldArgs& a, int bits, hipStream_t st) {
  return launch_out<4, true>(a, bits, st);
}

}  // namespace fgq
