// group_kernel.h -- FGQ layer with groups of 64 input channels on the int8
// matrix cores (gfx950), the per-group form of Sec. 4: 32-bit integer group sums,
// then one fp32 multiply-add by the group's scale per group.
//
// A group of 64 consecutive k is exactly two K slices of
// v_mfma_i32_32x32x32_i8, so for each group and each 32x32 block of
// (rows, channels) the matrix cores produce the exact int32 group sums
//   P[m][o] = sum_{k in g} t[o][k] * q[m][k]
// and the vector ALU folds them into the fp32 accumulator,
//   y[m][o] += alpha[o][g] * float(P[m][o]),
// with the output y * s_x stored once.  The rounding error is at most
// (K/64 + 1) fp32 roundings relative to s_x * sum_g alpha_g |P_g|.
//
// uint8 activations enter the signed instruction as q'' = 127 - q
// (q XOR 0x7F, padding reads 0 -> 127), and each group's block accumulation
// starts from -127 * sum_{k in g} t[o][k], which the matrix cores compute
// from a constant operand once per group and channel block, so the block
// result is exactly -P and the epilogue multiplies by -alpha.  uint4
// activations (0..15) need no offset.
//
// Staging of activations (LDS) follows the folded-scale kernel; see
// igemm.h.  The weights are read as the 2-bit codes (one 16-byte load per
// lane and step, a contiguous kilobyte per wave, see prepare.hip) and
// expanded to int8 in registers, one byte permute per four weights.
//
// The output kind is a template parameter (fp32 y, or 8-/4-bit codes of the
// next layer's activations); each kind is instantiated in a source file of
// its own (group.hip, group_q8.hip, group_q4.hip).
#pragma once

#include "igemm.h"
#include "epilogue.h"
#include "qcode.h"
#include "xexpand.h"

namespace fgq {

struct GroupArgs {
  ig::ActArgs x;
  const float* sx;
  const uint32_t* codes;  // [O32/32][Kp/128][64 lanes][4 words], see prepare.hip
  const float* alpha;    // [Kp/64][O32]
  float* y;
  uint8_t* qo;           // output codes (kOut 8 or 4)
  const float* oscale;   // their scale
  const float* res = nullptr;  // residual added before the ReLU (kOut 2)
  int32_t staged;        // epilogue through LDS (epi_staged)
  int32_t nks, O32, codes_bytes, alpha_bytes;
};

// One launcher per output kind: kOut = 0 (fp32 y), 8 or 4 (codes).
fgq_status launch_group_out_f32(const GroupArgs& a, int bits, hipStream_t st);
fgq_status launch_group_out_q8(const GroupArgs& a, int bits, hipStream_t st);
fgq_status launch_group_out_q4(const GroupArgs& a, int bits, hipStream_t st);
fgq_status launch_group_out_res(const GroupArgs& a, int bits, hipStream_t st);
fgq_status launch_group_out_res_q8(const GroupArgs& a, int bits, hipStream_t st);
fgq_status launch_group_out_res_q4(const GroupArgs& a, int bits, hipStream_t st);

namespace {

using namespace ig;

constexpr int kStepBytes = 64 * 16;  // codes of one channel tile, one 128-wide step

// Two workgroups may share a compute unit (at most 256 registers per lane):
// with two waves per SIMD, one wave's conversions and multiply-adds run
// while the other waits on its matrix instructions.
template <int kBits, int kNWO, int kNB, int kCM, int kOut>
__global__ __launch_bounds__(kThreads, 2) void group_conv_kernel(GroupArgs a) {
  constexpr int kNWM = 4 / kNWO;
  constexpr int kTO = 32 * kNWO;
  constexpr int kTM = kNWM * kNB * 32;
  using Stager = StagerFor<kBits, kTM, kCM>;
  constexpr int kStage = Stager::kStage;
  constexpr int kLds = 2 * kStage > EpiTile<kOut, kNWO>::kBytes ? 2 * kStage : EpiTile<kOut, kNWO>::kBytes;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLds];

  const int tid = threadIdx.x;
  const int lane = tid % 64, wave = tid / 64;
  const int wo = wave % kNWO, wm = wave / kNWO;
  const int tile = xcd_swizzle(blockIdx.x, a.x.n_otiles * a.x.n_mtiles);
  const int o0 = (tile % a.x.n_otiles) * kTO + 32 * wo;  // this wave's first channel
  const int m0 = (tile / a.x.n_otiles) * kTM;             // workgroup's first row

  const Buf wrs = make_buf(a.codes, a.codes_bytes, kSiteCodes, kBufFlags);
  const Buf ars = make_buf(a.alpha, a.alpha_bytes, kSiteAlpha, kBufFlags);
  const int nk = (a.x.K + kKT - 1) / kKT;
  const int wbase = (o0 / 32) * nk * kStepBytes + 16 * lane;
  // The group's alphas are the scalar offset, which the buffer range check
  // does not cover: lanes of a channel tile past the padded channel count
  // (O32) take an out-of-range vector offset, which reads zeros, instead of
  // addressing past the end of the buffer.
  const int abase = o0 + lane % 32 < a.O32 ? 4 * (o0 + lane % 32) : static_cast<int>(kOutOfRange);

  Stager xs;
  xs.init(a.x, m0, tid);

  // Codes and scales of one step (two groups).  The step is the scalar
  // offset, which the buffer range check does not cover, so a step past the
  // last is clamped to the last one (those loads are never used).
  v4i cring[2];
  float aring[2][2];
  auto load_w = [&](auto U, int ks) {
    constexpr int u = decltype(U)::value;
    ks = ks < nk ? ks : nk - 1;
    cring[u] = buf_load_b128(wrs, wbase, ks * kStepBytes);
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
      aring[u][blk] = __builtin_bit_cast(
          float, buf_load_b32(ars, abase, (2 * ks + blk) * a.O32 * 4));
  };

  v16f acc[kNB];
#pragma unroll
  for (int c = 0; c < kNB; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.0f;

  int afrag[kNB][4];
#pragma unroll
  for (int c = 0; c < kNB; ++c)
#pragma unroll
    for (int h = 0; h < 4; ++h) afrag[c][h] = lds_off(wm * kNB * 32 + 32 * c + lane % 32, 2 * h + lane / 32);

  const v4i kMinus127 = {static_cast<int>(0x81818181u), static_cast<int>(0x81818181u),
                         static_cast<int>(0x81818181u), static_cast<int>(0x81818181u)};
  const v16i kZero = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};

  auto compute = [&](int stage, const v4i& cw, const float (&al)[2]) {
    const unsigned char* base = lds + stage * kStage;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      const v4i w[2] = {expand_ternary16(static_cast<uint32_t>(cw[2 * blk])),
                        expand_ternary16(static_cast<uint32_t>(cw[2 * blk + 1]))};
      v4i xf[kNB][2];
#pragma unroll
      for (int c = 0; c < kNB; ++c)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          xf[c][h] = *reinterpret_cast<const v4i*>(base + afrag[c][2 * blk + h]);
      v16i init = kZero;
      if constexpr (kBits == 8) {
        init = __builtin_amdgcn_mfma_i32_32x32x32_i8(kMinus127, w[0], kZero, 0, 0, 0);
        init = __builtin_amdgcn_mfma_i32_32x32x32_i8(kMinus127, w[1], init, 0, 0, 0);
      }
      const float s = kBits == 8 ? -al[blk] : al[blk];
#pragma unroll
      for (int c = 0; c < kNB; ++c) {
        v16i p = __builtin_amdgcn_mfma_i32_32x32x32_i8(xf[c][0], w[0], init, 0, 0, 0);
        p = __builtin_amdgcn_mfma_i32_32x32x32_i8(xf[c][1], w[1], p, 0, 0, 0);
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[c][r] = fmaf(s, static_cast<float>(p[r]), acc[c][r]);
      }
    }
  };

  // Step ks: prefetch step ks+1, feed the matrix cores from LDS stage ks%2,
  // then publish the prefetched activations to the other stage.
  constexpr uint32_t kMask = 0x7F7F7F7Fu;  // q -> 127 - q
  auto step = [&](auto U, int ks) {
    constexpr int u = decltype(U)::value;
    // Activation loads first: the publish at the end of the step waits for
    // them, and the memory counter is in order, so weight loads issued
    // before them would be waited for too.
    xs.advance(a.x);
    xs.load(a.x);
    __builtin_amdgcn_sched_barrier(0);
    load_w(std::integral_constant<int, 1 - u>{}, ks + 1);
    compute(u, cring[u], aring[u]);
    __builtin_amdgcn_sched_barrier(0);  // the publish waits for the prefetch: keep it last
    xs.store(lds + (1 - u) * kStage, kMask);
    __syncthreads();
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  load_w(I0{}, 0);
  xs.load(a.x);
  xs.store(lds, kMask);
  __syncthreads();
  int ks = 0;
  for (; ks + 2 <= nk; ks += 2) {
    step(I0{}, ks);
    step(I1{}, ks + 1);
  }
  if (ks < nk) step(I0{}, ks);

  // ---- epilogue: lane holds rows m of channel o.
  const int o = o0 + lane % 32;
  const float sx = *a.sx;
  // locals: a byte store may alias anything, including the argument block
  const OutPtrs out{a.y, a.qo, a.x.M, a.x.O, a.res};
  const bool staged = a.staged != 0;
  with_out_scale<kOut>(a.oscale, [&](const QScale& qs, auto rcp) {
    constexpr bool kR = decltype(rcp)::value;
    auto val = [&](int c, int r) { return acc[c][r] * sx; };
    if (staged)
      store_staged<kOut, kNWO, kNB, kR>(lds, out, qs, m0, o0 - 32 * wo, wm, wo, tid, val);
    else
      store_direct<kOut, kNB, kR>(out, qs, m0 + wm * kNB * 32, o, lane, val);
  });
}

template <int kOut, int kBits, int kNWO, int kNB>
fgq_status launch_cfg(const GroupArgs& a0, hipStream_t st) {
  constexpr int kTO = 32 * kNWO, kTM = (4 / kNWO) * kNB * 32;
  GroupArgs a = a0;
  a.x.n_otiles = (a.x.O + kTO - 1) / kTO;
  a.x.n_mtiles = (a.x.M + kTM - 1) / kTM;
  const int64_t n = static_cast<int64_t>(a.x.n_otiles) * a.x.n_mtiles;
  if (n > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  if (a.x.C < kKT)
    hipLaunchKernelGGL((group_conv_kernel<kBits, kNWO, kNB, 1, kOut>), dim3(static_cast<uint32_t>(n)),
                       dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((group_conv_kernel<kBits, kNWO, kNB, 0, kOut>), dim3(static_cast<uint32_t>(n)),
                       dim3(kThreads), 0, st, a);
  return last_launch();
}

// Rows per wave: two 32-row blocks (kNB = 2) for every shape.  Measured on
// the benchmark and network layers, 32-row tiles (more weight traffic per
// matrix instruction) and 128-row tiles (one workgroup per compute unit,
// and register spills in the per-group kernel) were slower, and a tile
// count balance of ceil(tiles / CUs) * kNB never prefers kNB = 4 over 2.
template <int kOut, int kBits, int kNWO>
fgq_status launch_nwo(const GroupArgs& a, hipStream_t st) {
  return launch_cfg<kOut, kBits, kNWO, 2>(a, st);
}

template <int kOut, int kBits>
fgq_status launch_bits(const GroupArgs& a, hipStream_t st) {
  if (a.x.O > 64) return launch_nwo<kOut, kBits, 4>(a, st);
  if (a.x.O > 32) return launch_nwo<kOut, kBits, 2>(a, st);
  return launch_nwo<kOut, kBits, 1>(a, st);
}

template <int kOut>
fgq_status launch_out(const GroupArgs& a, int bits, hipStream_t st) {
  return bits == 8 ? launch_bits<kOut, 8>(a, st) : launch_bits<kOut, 4>(a, st);
}

}  // namespace
}  // namespace fgq
