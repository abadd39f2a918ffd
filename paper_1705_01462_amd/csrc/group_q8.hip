// group_q8.hip -- the per-group (G = 64) layer kernels that emit 8-bit
// codes of the next layer's activations.
#include "group_kernel.h"

namespace fgq {

fgq_status launch_group_out_q8(const GroupArgs& a, int bits, hipStream_t st) { return launch_out<8>(a, bits, st); }

}  // namespace fgq
