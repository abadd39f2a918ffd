// group.hip -- FGQ layer with groups of 64 input channels on the int8 matrix
// cores (gfx950), the per-group form of Sec. 4: 32-bit integer group sums,
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
// Staging of activations (LDS) and weights (fragment-ordered, straight to
// registers) follows fold.hip; see igemm.h.
#include "igemm.h"

namespace fgq {
namespace {

using namespace ig;

struct GroupArgs {
  ActArgs x;
  const float* sx;
  const int8_t* planes;  // [O32/32][Kp/64][2][64][16]
  const float* alpha;    // [Kp/64][O32]
  float* y;
  int32_t nks, O32, planes_bytes, alpha_bytes;
};

constexpr int kBlkBytes = 2 * 64 * 16;  // one channel tile, one group

// Two workgroups may share a compute unit (at most 256 registers per lane):
// with two waves per SIMD, one wave's conversions and multiply-adds run
// while the other waits on its matrix instructions.
template <int kBits, int kNWO, int kNB, int kCM>
__global__ __launch_bounds__(kThreads, 2) void group_conv_kernel(GroupArgs a) {
  constexpr int kNWM = 4 / kNWO;
  constexpr int kTO = 32 * kNWO;
  constexpr int kTM = kNWM * kNB * 32;
  using Stager = StagerFor<kBits, kTM, kCM>;
  constexpr int kStage = Stager::kStage;
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * kStage];

  const int tid = threadIdx.x;
  const int lane = tid % 64, wave = tid / 64;
  const int wo = wave % kNWO, wm = wave / kNWO;
  const int tile = xcd_swizzle(blockIdx.x, a.x.n_otiles * a.x.n_mtiles);
  const int o0 = (tile % a.x.n_otiles) * kTO + 32 * wo;  // this wave's first channel
  const int m0 = (tile / a.x.n_otiles) * kTM;             // workgroup's first row

  const __amdgpu_buffer_rsrc_t wrs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(a.planes), 0, a.planes_bytes, kBufFlags);
  const __amdgpu_buffer_rsrc_t ars =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.alpha), 0, a.alpha_bytes, kBufFlags);
  const int wbase = (o0 / 32) * a.nks * kBlkBytes + 16 * lane;
  const int abase = 4 * (o0 + lane % 32);

  Stager xs;
  xs.init(a.x, m0, tid);

  // Weights and scales of one step (two groups): loads past the last group
  // read zeros or another tile's weights and are never used.
  v4i wring[2][2][2];
  float aring[2][2];
  auto load_w = [&](auto U, int ks) {
    constexpr int u = decltype(U)::value;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      const int g = 2 * ks + blk;
#pragma unroll
      for (int h = 0; h < 2; ++h)
        wring[u][blk][h] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wbase + h * 1024, g * kBlkBytes, 0);
      aring[u][blk] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(ars, abase, g * a.O32 * 4, 0));
    }
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

  auto compute = [&](int stage, const v4i (&w)[2][2], const float (&al)[2]) {
    const unsigned char* base = lds + stage * kStage;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      v4i xf[kNB][2];
#pragma unroll
      for (int c = 0; c < kNB; ++c)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          xf[c][h] = *reinterpret_cast<const v4i*>(base + afrag[c][2 * blk + h]);
      v16i init = kZero;
      if constexpr (kBits == 8) {
        init = __builtin_amdgcn_mfma_i32_32x32x32_i8(kMinus127, w[blk][0], kZero, 0, 0, 0);
        init = __builtin_amdgcn_mfma_i32_32x32x32_i8(kMinus127, w[blk][1], init, 0, 0, 0);
      }
      const float s = kBits == 8 ? -al[blk] : al[blk];
#pragma unroll
      for (int c = 0; c < kNB; ++c) {
        v16i p = __builtin_amdgcn_mfma_i32_32x32x32_i8(xf[c][0], w[blk][0], init, 0, 0, 0);
        p = __builtin_amdgcn_mfma_i32_32x32x32_i8(xf[c][1], w[blk][1], p, 0, 0, 0);
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[c][r] = fmaf(s, static_cast<float>(p[r]), acc[c][r]);
      }
    }
  };

  // Step ks: prefetch step ks+1, feed the matrix cores from LDS stage ks%2,
  // then publish the prefetched activations to the other stage.
  const int nk = (a.x.K + kKT - 1) / kKT;
  constexpr uint32_t kMask = 0x7F7F7F7Fu;  // q -> 127 - q
  auto step = [&](auto U, int ks) {
    constexpr int u = decltype(U)::value;
    load_w(std::integral_constant<int, 1 - u>{}, ks + 1);
    xs.advance(a.x);
    xs.load(a.x);
    compute(u, wring[u], aring[u]);
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
  if (o >= a.x.O) return;
  const float sx = *a.sx;
#pragma unroll
  for (int c = 0; c < kNB; ++c) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * kNB * 32 + 32 * c + 8 * (r / 4) + 4 * (lane / 32) + (r % 4);
      if (m >= a.x.M) continue;
      __builtin_nontemporal_store(acc[c][r] * sx, a.y + static_cast<int64_t>(m) * a.x.O + o);
    }
  }
}

template <int kBits, int kNWO, int kNB>
fgq_status launch_cfg(const GroupArgs& a0, hipStream_t st) {
  constexpr int kTO = 32 * kNWO, kTM = (4 / kNWO) * kNB * 32;
  GroupArgs a = a0;
  a.x.n_otiles = (a.x.O + kTO - 1) / kTO;
  a.x.n_mtiles = (a.x.M + kTM - 1) / kTM;
  const int64_t n = static_cast<int64_t>(a.x.n_otiles) * a.x.n_mtiles;
  if (n > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  if (a.x.C < kKT)
    hipLaunchKernelGGL((group_conv_kernel<kBits, kNWO, kNB, 1>), dim3(static_cast<uint32_t>(n)),
                       dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((group_conv_kernel<kBits, kNWO, kNB, 0>), dim3(static_cast<uint32_t>(n)),
                       dim3(kThreads), 0, st, a);
  return last_launch();
}

// Rows per wave (kNB blocks of 32): the busiest compute unit does
// ceil(tiles / CUs) workgroups of kNB blocks per SIMD; among equal costs
// the smaller kNB wins (more waves to overlap).
template <int kBits, int kNWO>
fgq_status launch_nwo(const GroupArgs& a, hipStream_t st) {
  constexpr int kNWM = 4 / kNWO;
  const int64_t otiles = ceil_div(a.x.O, 32 * kNWO);
  int best = 2;
  int64_t best_cost = -1;
  for (int nb = 2; nb <= 4; ++nb) {
    const int64_t tiles = otiles * ceil_div(a.x.M, kNWM * nb * 32);
    const int64_t cost = ceil_div(tiles, device_cus()) * nb;
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best = nb;
    }
  }
  switch (best) {
    case 2: return launch_cfg<kBits, kNWO, 2>(a, st);
    case 3: return launch_cfg<kBits, kNWO, 3>(a, st);
    default: return launch_cfg<kBits, kNWO, 4>(a, st);
  }
}

template <int kBits>
fgq_status launch_bits(const GroupArgs& a, hipStream_t st) {
  if (a.x.O > 64) return launch_nwo<kBits, 4>(a, st);
  if (a.x.O > 32) return launch_nwo<kBits, 2>(a, st);
  return launch_nwo<kBits, 1>(a, st);
}

}  // namespace

bool group_supported(const ConvGeom& g, const uint8_t* q) {
  const PreparedLayout L = prepared_layout(g.O, g.K, g.G);
  return L.kind == kPrepGroup && ig::igemm_shape_ok(g, q) && L.O32 * L.Kp < (1LL << 31) &&
         4 * L.nks * L.O32 < (1LL << 31);
}

fgq_status launch_group_conv(const uint8_t* q, const float* sx, const void* prepared,
                             const ConvGeom& g, float* y, hipStream_t st) {
  const PreparedLayout L = prepared_layout(g.O, g.K, g.G);
  const char* base = static_cast<const char*>(prepared);
  GroupArgs a;
  ig::fill_act_args(g, q, &a.x);
  a.sx = sx;
  a.planes = reinterpret_cast<const int8_t*>(base + L.planes_off);
  a.alpha = reinterpret_cast<const float*>(base + L.alpha_off);
  a.y = y;
  a.nks = static_cast<int32_t>(L.nks);
  a.O32 = static_cast<int32_t>(L.O32);
  a.planes_bytes = static_cast<int32_t>(L.O32 * L.Kp);
  a.alpha_bytes = static_cast<int32_t>(4 * L.nks * L.O32);
  return g.bits == 8 ? launch_bits<8>(a, st) : launch_bits<4>(a, st);
}

}  // namespace fgq
