// fold_res.hip -- the folded-scale layer kernels whose fp32 output takes a
// residual block's shortcut addition and ReLU.
#include "fold_kernel.h"

namespace fgq {

fgq_status launch_fold_out_res(const FoldArgs& a, int bits, hipStream_t st) { return launch_out<2>(a, bits, st); }

}  // namespace fgq
