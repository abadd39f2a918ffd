// group_res_q4.hip -- the per-group (G = 64) layer kernels whose fp32 output takes a
// residual block's shortcut addition and ReLU and that also write its
// 4-bit codes (the next block's input).
#include "group_kernel.h"

namespace fgq {

fgq_status launch_group_out_res_q4(const GroupArgs& a, int bits, hipStream_t st) { return launch_out<2 | 4>(a, bits, st); }

}  // namespace fgq
