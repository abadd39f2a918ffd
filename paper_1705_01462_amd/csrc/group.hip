// group.hip -- per-group (G = 64) FGQ layer: host entry (shape support,
// argument set-up from the prepared buffer) and the fp32-output instantiation.
#include "group_kernel.h"

namespace fgq {

bool group_supported(const ConvGeom& g, const uint8_t* q) {
  const PreparedLayout L = prepared_layout(g.O, g.K, g.G);
  return L.kind == kPrepGroup && ig::igemm_shape_ok(g, q) && L.O32 * L.Kp / 4 < (1LL << 31) &&
         4 * L.nks * L.O32 < (1LL << 31);
}

fgq_status launch_group_conv(const uint8_t* q, const float* sx, const void* prepared,
                             const ConvGeom& g, const LayerOut& out, hipStream_t st) {
  const PreparedLayout L = prepared_layout(g.O, g.K, g.G);
  const char* base = static_cast<const char*>(prepared);
  GroupArgs a;
  ig::fill_act_args(g, q, &a.x);
  a.sx = sx;
  a.codes = reinterpret_cast<const uint32_t*>(base + L.planes_off);
  a.alpha = reinterpret_cast<const float*>(base + L.alpha_off);
  a.y = out.y;
  a.qo = out.q;
  a.oscale = out.scale;
  a.res = out.res;
  a.staged = ig::epi_staged(out.bits, g.O, out.y, out.q, out.res);
  a.nks = static_cast<int32_t>(L.nks);
  a.O32 = static_cast<int32_t>(L.O32);
  a.codes_bytes = static_cast<int32_t>(L.O32 * L.Kp / 4);
  a.alpha_bytes = static_cast<int32_t>(4 * L.nks * L.O32);
  switch (out.bits) {
    case 0: return launch_group_out_f32(a, g.bits, st);
    case 2: return launch_group_out_res(a, g.bits, st);
    case 2 | 8: return launch_group_out_res_q8(a, g.bits, st);
    case 2 | 4: return launch_group_out_res_q4(a, g.bits, st);
    case 8: return launch_group_out_q8(a, g.bits, st);
    default: return launch_group_out_q4(a, g.bits, st);
  }
}

fgq_status launch_group_out_f32(const GroupArgs& a, int bits, hipStream_t st) { return launch_out<0>(a, bits, st); }

}  // namespace fgq
