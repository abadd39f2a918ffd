// fold_dfp_res_q4.hip -- the fixed-point-scale layer kernels whose fp32 output
// takes a residual block's shortcut addition and ReLU and that also write
// its 4-bit codes (the next block's input).
#include "fold_kernel.h"

namespace fgq {

fgq_status launch_fold_dfp_out_res_q4(const FoldArgs& a, int bits, hipStream_t st) {
  return launch_out<2 | 4, true>(a, bits, st);
}

}  // namespace fgq
