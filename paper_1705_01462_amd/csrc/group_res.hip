// group_res.hip -- the per-group (G = 64) layer kernels whose fp32 output
// takes a residual block's shortcut addition and ReLU.
#include "group_kernel.h"

namespace fgq {

fgq_status launch_group_out_res(const GroupArgs& a, int bits, hipStream_t st) { return launch_out<2>(a, bits, st); }

}  // namespace fgq
