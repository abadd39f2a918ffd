// fold_rows.hip -- host entry of the row-walking folded kernel (fold_rows.h).
#include "fold_rows.h"

namespace fgq {

// K <= 128 (one resident step), O > 64 (four channel waves, 128-channel
// tiles, 64-row tiles) and at least two row tiles per workgroup of a grid
// of two workgroups per compute unit.
bool fold_rows_eligible(const FoldArgs& a) {
  if (a.splits != 1 || a.x.K > ig::kKT || ig::c_mode(a.x.C) > 1 || a.x.O <= 64) return false;
  const int64_t tiles = ceil_div(a.x.O, 128) * ceil_div(a.x.M, 64);
  return tiles >= 4LL * ig::device_cus();
}

fgq_status launch_fold_rows(const FoldArgs& a, int bits, int out_bits, hipStream_t st) {
  switch (out_bits) {
    case 0: return launch_rows<0>(a, bits, st);
    case 2: return launch_rows<2>(a, bits, st);
    case 2 | 8: return launch_rows<2 | 8>(a, bits, st);
    case 2 | 4: return launch_rows<2 | 4>(a, bits, st);
    case 8: return launch_rows<8>(a, bits, st);
    default: return launch_rows<4>(a, bits, st);
  }
}

}  // namespace fgq
