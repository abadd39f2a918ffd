// fold_dfp_res.hip -- the fixed-point-scale layer kernels whose fp32 output
// takes a residual block's shortcut addition and ReLU.
#include "fold_kernel.h"

namespace fgq {

fgq_status launch_fold_dfp_out_res(const FoldArgs& a, int bits, hipStream_t st) {
  return launch_out<2, true>(a, bits, st);
}

}  // namespace fgq
