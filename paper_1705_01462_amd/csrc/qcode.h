// qcode.h -- the unsigned activation code of one value (Sec. 4: activations
// quantized with one scale per tensor), shared by the quantize kernel and
// the convolution epilogues that emit quantized activations:
//   code = min(max(rint(v / s), 0), qmax), qmax = 2^bits - 1,
// with the correctly rounded quotient v / s and rint rounding half to even,
// so that codes are reproducible bit for bit; NaN maps to 0.
//
// The quotient is formed from the correctly rounded reciprocal y = 1/s,
// taken once per scale: q0 = v*y is within one ulp of v/s, the residual
// v - q0*s is exact in one fused multiply-add, and q0 + (v - q0*s)*y rounded
// once is the correctly rounded quotient (Markstein's theorem on a single
// correction step, valid while s, y and the quotient are normal numbers).
// q0 is first clamped to +-2^24: a quotient that large saturates the code
// either way, and the clamp keeps the residual finite when v*y overflows
// (an infinite v still gives an infinite, hence saturated, quotient).  When
// s or y is not a normal number, plain division; that choice is uniform
// over a launch and is made once, outside the loops over values
// (with_rcp).
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

namespace fgq {

struct QScale {
  float s, y, qmax;
  bool rcp;
};

__device__ inline QScale make_qscale(float s, int bits) {
#pragma clang fp contract(off)
  QScale c;
  c.s = s;
  c.y = 1.0f / s;
  c.qmax = bits == 8 ? 255.0f : 15.0f;
  const float kMinNormal = 1.17549435e-38f;
  // the same in every lane: made a scalar, so that branches on it are uniform
  c.rcp = __builtin_amdgcn_readfirstlane(
              static_cast<int>(s >= kMinNormal && c.y >= kMinNormal && c.y < __builtin_huge_valf())) != 0;
  return c;
}

template <bool kRcp>
__device__ inline unsigned qcode(float v, const QScale& c) {
#pragma clang fp contract(off)
  float q;
  if constexpr (kRcp) {
    const float q0 = fminf(fmaxf(v * c.y, -16777216.0f), 16777216.0f);
    q = fmaf(fmaf(-q0, c.s, v), c.y, q0);
  } else {
    q = v / c.s;
  }
  const float r = fminf(fmaxf(rintf(q), 0.0f), c.qmax);  // NaN -> 0
  return static_cast<unsigned>(r);
}

// f(std::true_type{}) when the scale admits the reciprocal form, else
// f(std::false_type{}); f passes the flag on to qcode / emit_out.
template <class F>
__device__ inline void with_rcp(const QScale& c, F&& f) {
  if (c.rcp)
    f(std::true_type{});
  else
    f(std::false_type{});
}

// Output kinds of the layer kernels, as bit sets: 0 = fp32 output; 8 or 4 =
// codes (8 or 4 bits) of the output instead; 2 = fp32 output with a
// residual added before a ReLU; 2 | 8, 2 | 4 = that output and also its
// codes.  (Kind 1, split-K partial sums, never reaches an epilogue.)
constexpr bool out_res(int kind) { return kind != 1 && (kind & 2) != 0; }
constexpr bool out_f32(int kind) { return kind == 0 || out_res(kind); }
constexpr int out_code_bits(int kind) { return kind == 1 ? 0 : (kind & 12); }

// The fused shortcut addition and ReLU of output kind 2: max(v + r, 0), the
// sum rounded once (a NaN sum stays NaN).  No contraction: v is often a
// product, and an addition fused with it would round differently from the
// layer's own fp32 output plus r.
__device__ inline float add_relu(float v, float r) {
#pragma clang fp contract(off)
  const float s = v + r;
  return s < 0.0f ? 0.0f : s;
}

// One output value of a layer, at element index e = m*O + o of n = M*O, by
// output kind: the residual and ReLU first where the kind has them
// (v = max(v + res[e], 0)), then v stored as fp32 to y where it has an
// fp32 output, and its code to q where it has codes: one byte (8 bits), or
// two codes per byte (4 bits; the lanes holding channels o and o^1 must
// call together and the even one writes).  All stores are non-temporal: the
// output is written once, and streaming it out leaves no dirty lines in the
// per-XCD L2 caches for the end of the kernel to write back.
template <int kOut, bool kRcp = true>
__device__ inline void emit_out(float* y, uint8_t* q, const QScale& qs, int64_t e, int64_t n, int o, float v,
                                const float* res = nullptr) {
  constexpr int kCode = out_code_bits(kOut);
  if constexpr (out_res(kOut)) {
    if (check_store(kSiteStoreY, e, 1, n)) v = add_relu(v, __builtin_nontemporal_load(res + e));
  }
  if constexpr (out_f32(kOut)) {
    if (check_store(kSiteStoreY, e, 1, n)) __builtin_nontemporal_store(v, y + e);
  }
  if constexpr (kCode == 8) {
    if (check_store(kSiteStoreY, e, 1, n)) __builtin_nontemporal_store(static_cast<uint8_t>(qcode<kRcp>(v, qs)), q + e);
  } else if constexpr (kCode == 4) {
    const unsigned c = qcode<kRcp>(v, qs);
    const unsigned other = static_cast<unsigned>(__builtin_amdgcn_mov_dpp(static_cast<int>(c), 0xB1, 0xF, 0xF, false));
    if ((o & 1) == 0 && check_store(kSiteStoreY, e >> 1, 1, (n + 1) / 2))
      __builtin_nontemporal_store(static_cast<uint8_t>(c | (other << 4)), q + (e >> 1));
  }
}

// The store loop of a layer epilogue, run as f(qs, rcp) with the output
// kind's scale: for codes, qs is the scale read from `scale` and rcp the
// reciprocal-form flag as a type (see with_rcp); for fp32 output neither is
// used.
template <int kOut, class F>
__device__ inline void with_out_scale(const float* scale, F&& f) {
  if constexpr (out_code_bits(kOut) == 0) {
    f(QScale{}, std::true_type{});
  } else {
    const QScale qs = make_qscale(*scale, out_code_bits(kOut));
    with_rcp(qs, [&](auto rcp) { f(qs, rcp); });
  }
}

}  // namespace fgq
