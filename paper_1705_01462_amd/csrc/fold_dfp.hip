// fold_dfp.hip -- the layer with fixed-point group scales (dfp.hip) on the
// folded kernel with one weight plane: host entry and the fp32-output
// instantiation.
#include "fold_kernel.h"

namespace fgq {

bool fold_dfp_supported(const ConvGeom& g, const uint8_t* q) {
  const PreparedLayout L = prepared_layout_dfp(g.O, g.K, g.G);
  return g.K <= kFoldMaxK && ig::igemm_shape_ok(g, q, /*tiny_c=*/true) && L.O32 * L.Kp < (1LL << 31);
}

fgq_status launch_fold_dfp_conv(const uint8_t* q, const float* sx, const void* prepared,
                                const ConvGeom& g, const LayerOut& out, hipStream_t st) {
  const PreparedLayout L = prepared_layout_dfp(g.O, g.K, g.G);
  const char* base = static_cast<const char*>(prepared);
  FoldArgs a;
  ig::fill_act_args(g, q, &a.x);
  a.sx = sx;
  a.planes = reinterpret_cast<const int8_t*>(base + L.planes_off);
  a.bias = reinterpret_cast<const int32_t*>(base + L.bias_off);
  a.scale = nullptr;
  a.y = out.y;
  a.qo = out.q;
  a.oscale = out.scale;
  a.fl = reinterpret_cast<const int32_t*>(base);
  a.part = nullptr;
  a.splits = 1;
  a.steps_per_split = 1 << 30;
  a.res = out.res;
  a.staged = ig::epi_staged(out.bits, g.O, out.y, out.q, out.res);
  a.nks = static_cast<int32_t>(L.nks);
  a.planes_bytes = static_cast<int32_t>(L.O32 * L.Kp);
  a.xg = 0;  // the one-plane kernel reads the plane (see launch_out)
  switch (out.bits) {
    case 0: return launch_fold_dfp_out_f32(a, g.bits, st);
    case 2: return launch_fold_dfp_out_res(a, g.bits, st);
    case 2 | 8: return launch_fold_dfp_out_res_q8(a, g.bits, st);
    case 2 | 4: return launch_fold_dfp_out_res_q4(a, g.bits, st);
    case 8: return launch_fold_dfp_out_q8(a, g.bits, st);
    default: return launch_fold_dfp_out_q4(a, g.bits, st);
  }
}

fgq_status launch_fold_dfp_out_f32(const FoldArgs& a, int bits, hipStream_t st) {
  return launch_out<0, true>(a, bits, st);
}

fgq_status launch_fold_dfp_splitk(const uint8_t* q, const float* sx, const void* prepared, const ConvGeom& g,
                                  const LayerOut& out, int32_t splits, int32_t steps_per_split, int32_t* ws,
                                  hipStream_t st) {
  const PreparedLayout L = prepared_layout_dfp(g.O, g.K, g.G);
  const char* base = static_cast<const char*>(prepared);
  FoldArgs a;
  ig::fill_act_args(g, q, &a.x);
  a.sx = sx;
  a.planes = reinterpret_cast<const int8_t*>(base + L.planes_off);
  a.bias = reinterpret_cast<const int32_t*>(base + L.bias_off);
  a.scale = nullptr;
  a.y = nullptr;
  a.qo = nullptr;
  a.oscale = nullptr;
  a.fl = reinterpret_cast<const int32_t*>(base);
  a.part = ws;
  a.splits = splits;
  a.steps_per_split = steps_per_split;
  a.staged = 0;
  a.nks = static_cast<int32_t>(L.nks);
  a.planes_bytes = static_cast<int32_t>(L.O32 * L.Kp);
  a.xg = 0;
  fgq_status rc = launch_fold_dfp_part(a, g.bits, st);
  if (rc != FGQ_OK) return rc;
  return launch_splitk_reduce(ws, splits, /*dfp=*/true, g.M, g.O, sx, nullptr, a.fl, out, st);
}

}  // namespace fgq
