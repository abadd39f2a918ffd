// fold.hip -- folded-scale FGQ layer: host entry (shape support, argument
// set-up from the prepared buffer) and the fp32-output instantiation.
#include "fold_kernel.h"

namespace fgq {

bool fold_supported(const ConvGeom& g, const uint8_t* q) {
  const PreparedLayout L = prepared_layout(g.O, g.K, g.G);
  return L.kind == kPrepFold && g.K <= kFoldMaxK && ig::igemm_shape_ok(g, q, /*tiny_c=*/true) &&
         3 * L.O32 * L.Kp < (1LL << 31);
}

fgq_status launch_fold_conv(const uint8_t* q, const float* sx, const void* prepared,
                            const ConvGeom& g, const LayerOut& out, hipStream_t st) {
  const PreparedLayout L = prepared_layout(g.O, g.K, g.G);
  const char* base = static_cast<const char*>(prepared);
  FoldArgs a;
  ig::fill_act_args(g, q, &a.x);
  a.sx = sx;
  a.planes = reinterpret_cast<const int8_t*>(base + L.planes_off);
  a.bias = reinterpret_cast<const int32_t*>(base + L.bias_off);
  a.scale = reinterpret_cast<const float*>(base + L.scale_off);
  a.y = out.y;
  a.qo = out.q;
  a.oscale = out.scale;
  a.fl = nullptr;
  a.part = nullptr;
  a.splits = 1;
  a.steps_per_split = 1 << 30;
  a.res = out.res;
  a.staged = ig::epi_staged(out.bits, g.O, out.y, out.q, out.res);
  a.nks = static_cast<int32_t>(L.nks);
  a.planes_bytes = static_cast<int32_t>(3 * L.O32 * L.Kp);
  set_codes_operand(a, g.G, base, L, 3);
  if (fold_rows_eligible(a)) return launch_fold_rows(a, g.bits, out.bits, st);
  switch (out.bits) {
    case 0: return launch_fold_out_f32(a, g.bits, st);
    case 2: return launch_fold_out_res(a, g.bits, st);
    case 2 | 8: return launch_fold_out_res_q8(a, g.bits, st);
    case 2 | 4: return launch_fold_out_res_q4(a, g.bits, st);
    case 8: return launch_fold_out_q8(a, g.bits, st);
    default: return launch_fold_out_q4(a, g.bits, st);
  }
}

fgq_status launch_fold_out_f32(const FoldArgs& a, int bits, hipStream_t st) { return launch_out<0>(a, bits, st); }

fgq_status launch_fold_splitk(const uint8_t* q, const float* sx, const void* prepared, const ConvGeom& g,
                              const LayerOut& out, int32_t splits, int32_t steps_per_split, int32_t* ws,
                              hipStream_t st) {
  const PreparedLayout L = prepared_layout(g.O, g.K, g.G);
  const char* base = static_cast<const char*>(prepared);
  FoldArgs a;
  ig::fill_act_args(g, q, &a.x);
  a.sx = sx;
  a.planes = reinterpret_cast<const int8_t*>(base + L.planes_off);
  a.bias = reinterpret_cast<const int32_t*>(base + L.bias_off);
  a.scale = reinterpret_cast<const float*>(base + L.scale_off);
  a.y = nullptr;
  a.qo = nullptr;
  a.oscale = nullptr;
  a.fl = nullptr;
  a.part = ws;
  a.splits = splits;
  a.steps_per_split = steps_per_split;
  a.staged = 0;
  a.nks = static_cast<int32_t>(L.nks);
  a.planes_bytes = static_cast<int32_t>(3 * L.O32 * L.Kp);
  a.xg = 0;
  fgq_status rc = launch_fold_part(a, g.bits, st);
  if (rc != FGQ_OK) return rc;
  return launch_splitk_reduce(ws, splits, /*dfp=*/false, g.M, g.O, sx, a.scale, nullptr, out, st);
}

}  // namespace fgq
