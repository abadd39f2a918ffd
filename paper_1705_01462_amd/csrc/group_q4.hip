// group_q4.hip -- the per-group (G = 64) layer kernels that emit 4-bit
// codes of the next layer's activations.
#include "group_kernel.h"

namespace fgq {

fgq_status launch_group_out_q4(const GroupArgs& a, int bits, hipStream_t st) { return launch_out<4>(a, bits, st); }

}  // namespace fgq
