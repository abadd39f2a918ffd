// fold.hip -- folded-scale FGQ layer on the int8 matrix cores (gfx950).
//
// With the per-group scales folded into three int8 digit planes (see
// prepare.hip), the layer is three exact int8 GEMMs sharing one activation
// operand:
//   S_j[o][m] = sum_k plane_j[o][k] * q'[m][k],   q' = q ^ 0x80 (uint8) or q (uint4)
//   y[m][o]   = sum_j (S_j + bias_j[o]) * (s_x * 2^-E_o * 255^j)
// The integer sums are exact (|S_j| < 2^31 for K < 2^17); the combination
// is three fp32 conversions and fused multiply-adds per output.
//
// Implicit GEMM: row m = (b, ho, wo), k = (r*S + s)*C + c, so a 16-element
// piece of k (C % 16 == 0) is 16 consecutive channels of one input pixel.
//
// Work split.  A 256-thread workgroup owns a tile of output rows x output
// channels and walks K in steps of 64 (one v_mfma_i32_16x16x64_i8 K).  Its
// four waves are kNWO (channels) x 4/kNWO (rows); each wave owns 32
// channels x kMB*16 rows, i.e. 2 x kMB 16x16 blocks per digit plane.
//  * Weights (the 16-row MFMA operand) go straight from memory (L2: every
//    workgroup reads the same few hundred KB) into registers, one step
//    ahead; no two waves of a workgroup share them.
//  * Activations (the 16-column operand) are gathered into LDS once per
//    workgroup per step (double-buffered) and read by every wave that
//    shares those rows.
// A lane's four accumulators are four consecutive channels of one output
// row, so each fp32 result leaves as one 16-byte store.  Workgroups are
// numbered so that consecutive row tiles land on one XCD (shared halos in
// that XCD's L2).  All in-loop index arithmetic is 32-bit and incremental.
#include <type_traits>

#include "fgq_internal.h"

namespace fgq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kKT = 64;            // K per step
constexpr int kLdsRow = kKT + 16;  // bytes per LDS row; 80 spreads 16-byte reads over the banks

struct FoldArgs {
  const uint8_t* q;
  const float* sx;
  const int8_t* planes;
  const int32_t* bias;
  const float* scale;
  float* y;
  int32_t M, K, O, Kp;
  int32_t H, W, C, R, S, Ho, Wo, sh, sw, ph, pw;
  int32_t n_otiles, n_mtiles;
};

// Unpack 16 four-bit values (8 bytes, element 2i in the low nibble) to 16
// bytes in element order.
__device__ inline v4i unpack_u4x16(uint2 v) {
  const uint32_t lo0 = v.x & 0x0F0F0F0Fu, hi0 = (v.x >> 4) & 0x0F0F0F0Fu;
  const uint32_t lo1 = v.y & 0x0F0F0F0Fu, hi1 = (v.y >> 4) & 0x0F0F0F0Fu;
  v4i r;
  r.x = static_cast<int>(__builtin_amdgcn_perm(hi0, lo0, 0x05010400u));
  r.y = static_cast<int>(__builtin_amdgcn_perm(hi0, lo0, 0x07030602u));
  r.z = static_cast<int>(__builtin_amdgcn_perm(hi1, lo1, 0x05010400u));
  r.w = static_cast<int>(__builtin_amdgcn_perm(hi1, lo1, 0x07030602u));
  return r;
}

__device__ inline int xcd_swizzle(int bid, int n) {
  // Hardware places workgroup i on XCD i % 8: give each XCD a contiguous
  // run of logical tiles.
  const int x = bid % 8, qn = n / 8, rn = n % 8;
  return x * qn + (x < rn ? x : rn) + bid / 8;
}

template <int kBits, int kNWO, int kMB, bool kSmallC>
__global__ __launch_bounds__(kThreads, 1) void fold_conv_kernel(FoldArgs a) {
  constexpr int kNWM = 4 / kNWO;
  constexpr int kTO = 32 * kNWO;
  constexpr int kTM = kNWM * kMB * 16;
  constexpr int kPieces = kTM * 4;  // 16-byte pieces of one activation step
  constexpr int kXP = (kPieces + kThreads - 1) / kThreads;
  // Pieces past the tile (when kTM*4 is not a multiple of 256) are written
  // to spare rows after the tile so that every store is unconditional.
  constexpr int kStage = (kTM + (kXP * kThreads - kPieces) / 4) * kLdsRow;
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * kStage];

  const int tid = threadIdx.x;
  const int lane = tid % 64, wave = tid / 64;
  const int wo = wave % kNWO, wm = wave / kNWO;
  const int tile = xcd_swizzle(blockIdx.x, a.n_otiles * a.n_mtiles);
  const int o0 = (tile % a.n_otiles) * kTO + 32 * wo;  // this wave's first channel
  const int m0 = (tile / a.n_otiles) * kTM;             // workgroup's first row

  // ---- weight fragment pointers: lane supplies channel o0+16b+lane%16,
  // k-slot 16*(lane/16) of each step.  Channels past O read channel O-1
  // (their results are never stored).
  const int8_t* wp[3][2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    int o = o0 + 16 * b + lane % 16;
    o = o < a.O ? o : a.O - 1;
#pragma unroll
    for (int j = 0; j < 3; ++j)
      wp[j][b] = a.planes + (static_cast<int64_t>(j) * a.O + o) * a.Kp + 16 * (lane / 16);
  }

  // ---- activation pieces owned by this thread: piece p = tid + 256*i is
  // row p/4 of the tile, k-slot 16*(p%4) = 16*(tid%4) of each step.
  const int sub = tid % 4;
  int rowbase[kXP], hi0[kXP], wi0[kXP];
  bool rowok[kXP];
#pragma unroll
  for (int i = 0; i < kXP; ++i) {
    const int p = tid + kThreads * i;
    const int m = m0 + p / 4;
    rowok[i] = (p < kPieces) && (m < a.M);
    const int mm = rowok[i] ? m : 0;
    const int wo_ = mm % a.Wo;
    const int t = mm / a.Wo;
    const int ho = t % a.Ho;
    const int b = t / a.Ho;
    hi0[i] = ho * a.sh - a.ph;
    wi0[i] = wo_ * a.sw - a.pw;
    rowbase[i] = (b * a.H + hi0[i]) * a.W + wi0[i];
  }
  // tap state (r, s, c) of k = step*64 + 16*sub, advanced incrementally
  int tr, ts, tc, tk = 16 * sub;
  {
    const int rs = tk / a.C;
    tc = tk - rs * a.C;
    ts = rs % a.S;
    tr = rs / a.S;
  }
  auto advance_tap = [&]() {
    tk += kKT;
    if constexpr (kSmallC) {  // C in {16, 32, 48}: several taps per step
      const int t = ts + (tc + kKT) / a.C;
      tc = (tc + kKT) % a.C;
      tr += t / a.S;
      ts = t % a.S;
    } else {                  // C >= 64: at most one tap boundary per step
      tc += kKT;
      const bool wrap = tc >= a.C;
      tc = wrap ? tc - a.C : tc;
      const int t = ts + (wrap ? 1 : 0);
      const bool wrap2 = t == a.S;
      ts = wrap2 ? 0 : t;
      tr += wrap2 ? 1 : 0;
    }
  };

  // Loads are unconditional (out-of-range pieces read the tensor's first
  // bytes); the zero select, the uint8 offset and the uint4 unpack happen
  // when the piece is written to LDS, so nothing waits on a load before the
  // matrix-core work of the step has been issued.
  typedef typename std::conditional<kBits == 8, v4i, uint2>::type raw_t;
  raw_t xraw[3][kXP];
  bool xok[3][kXP];
  auto load_x = [&](auto U) {
    constexpr int u = decltype(U)::value;
#pragma unroll
    for (int i = 0; i < kXP; ++i) {
      const int hi = hi0[i] + tr, wi = wi0[i] + ts;
      const bool ok = rowok[i] && tk < a.K && hi >= 0 && hi < a.H && wi >= 0 && wi < a.W;
      const int64_t e = ok ? static_cast<int64_t>(rowbase[i] + tr * a.W + ts) * a.C + tc : 0;
      xraw[u][i] = *reinterpret_cast<const raw_t*>(a.q + (kBits == 8 ? e : e / 2));
      xok[u][i] = ok;
    }
  };
  auto store_x = [&](auto U, int stage) {
    constexpr int u = decltype(U)::value;
    unsigned char* base = lds + stage * kStage;
#pragma unroll
    for (int i = 0; i < kXP; ++i) {
      const int p = tid + kThreads * i;
      v4i v;
      if constexpr (kBits == 8) {
        const int x = static_cast<int>(0x80808080u);
        v = xraw[u][i];
        if (!xok[u][i]) v = v4i{0, 0, 0, 0};
        v.x ^= x; v.y ^= x; v.z ^= x; v.w ^= x;  // q - 128; padding reads -128
      } else {
        v = xok[u][i] ? unpack_u4x16(xraw[u][i]) : v4i{0, 0, 0, 0};
      }
      *reinterpret_cast<v4i*>(base + (p / 4) * kLdsRow + 16 * (p % 4)) = v;
    }
  };

  v4i acc[3][2][kMB];
#pragma unroll
  for (int j = 0; j < 3; ++j)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int c = 0; c < kMB; ++c) acc[j][b][c] = v4i{0, 0, 0, 0};

  const int nk = (a.K + kKT - 1) / kKT;
  const int xrow0 = wm * kMB * 16 + lane % 16, xslot = 16 * (lane / 16);
  const unsigned char* xfrag = lds + xrow0 * kLdsRow + xslot;
  auto compute = [&](int stage, const v4i (&w)[3][2]) {
    const unsigned char* base = xfrag + stage * kStage;
    v4i xf[kMB];
#pragma unroll
    for (int c = 0; c < kMB; ++c) xf[c] = *reinterpret_cast<const v4i*>(base + 16 * c * kLdsRow);
#pragma unroll
    for (int c = 0; c < kMB; ++c)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int j = 0; j < 3; ++j)
          acc[j][b][c] = __builtin_amdgcn_mfma_i32_16x16x64_i8(w[j][b], xf[c], acc[j][b][c], 0, 0, 0);
    // Issue every fragment read first (distinct registers), then the
    // matrix instructions, so LDS latency is paid once per step.
#pragma unroll
    for (int c = 0; c < kMB; ++c) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 6 * kMB, 0);
  };

  // Software pipeline, two steps deep: step ks issues the loads of step
  // ks+2 (weights into ring slot (ks+2)%3, activations into registers),
  // feeds the matrix cores with LDS stage ks%2 and ring slot ks%3, then
  // publishes the activations of step ks+1 (loaded a step earlier) to the
  // other LDS stage.  Prefetches past the last step reload the last step's
  // weights and read no activations, so no load needs a branch.  The loop
  // is unrolled by 3 so that every ring index is a compile-time constant.
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  v4i wring[3][3][2];
  const int klast = (nk - 1) * kKT;
  auto load_w_step = [&](auto U, int ks) {
    constexpr int u = decltype(U)::value;
    const int kc = ks * kKT < klast ? ks * kKT : klast;
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
      for (int b = 0; b < 2; ++b) wring[u][j][b] = *reinterpret_cast<const v4i*>(wp[j][b] + kc);
  };
  auto step = [&](auto U, int ks) {
    constexpr int u = decltype(U)::value;
    constexpr int u2 = (u + 2) % 3, u1 = (u + 1) % 3;
    load_w_step(std::integral_constant<int, u2>{}, ks + 2);
    advance_tap();
    load_x(std::integral_constant<int, u2>{});
    __builtin_amdgcn_sched_barrier(0);  // prefetch issued before the matrix work
    compute(ks & 1, wring[u]);
    __builtin_amdgcn_sched_barrier(0);  // publish (which waits) after it
    store_x(std::integral_constant<int, u1>{}, (ks + 1) & 1);
    __syncthreads();
  };

  load_w_step(I0{}, 0);
  load_x(I0{});
  load_w_step(I1{}, 1);
  advance_tap();
  load_x(I1{});
  store_x(I0{}, 0);
  __syncthreads();
  int ks = 0;
  for (; ks + 3 <= nk; ks += 3) {
    step(I0{}, ks);
    step(I1{}, ks + 1);
    step(I2{}, ks + 2);
  }
  if (ks < nk) step(I0{}, ks);
  if (ks + 1 < nk) step(I1{}, ks + 1);

  // ---- epilogue: lane holds channels ob..ob+3 of row m.
  const float sx = *a.sx;
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int ob = o0 + 16 * b + 4 * (lane / 16);
    float c0[4], c1[4], c2[4];
    int32_t b0[4], b1[4], b2[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int o = ob + r;
      const bool ok = o < a.O;
      const float s0 = ok ? sx * a.scale[o] : 0.0f;
      c0[r] = s0;
      c1[r] = s0 * 255.0f;
      c2[r] = s0 * 65025.0f;
      if (kBits == 8 && ok) {
        b0[r] = a.bias[o];
        b1[r] = a.bias[a.O + o];
        b2[r] = a.bias[2 * a.O + o];
      } else {
        b0[r] = b1[r] = b2[r] = 0;
      }
    }
#pragma unroll
    for (int c = 0; c < kMB; ++c) {
      const int m = m0 + wm * kMB * 16 + 16 * c + lane % 16;
      if (m >= a.M) continue;
      float out[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float f2 = static_cast<float>(acc[2][b][c][r] + b2[r]);
        const float f1 = static_cast<float>(acc[1][b][c][r] + b1[r]);
        const float f0 = static_cast<float>(acc[0][b][c][r] + b0[r]);
        out[r] = fmaf(f2, c2[r], fmaf(f1, c1[r], f0 * c0[r]));
      }
      float* dst = a.y + static_cast<int64_t>(m) * a.O + ob;
      if (ob + 3 < a.O && (a.O % 4) == 0) {
        const v4f v = {out[0], out[1], out[2], out[3]};
        __builtin_nontemporal_store(v, reinterpret_cast<v4f*>(dst));
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (ob + r < a.O) dst[r] = out[r];
      }
    }
  }
}

template <int kBits, int kNWO, int kMB>
fgq_status launch_cfg(const FoldArgs& a0, hipStream_t st) {
  const bool small_c = a0.C < kKT;
  constexpr int kTO = 32 * kNWO, kTM = (4 / kNWO) * kMB * 16;
  FoldArgs a = a0;
  a.n_otiles = (a.O + kTO - 1) / kTO;
  a.n_mtiles = (a.M + kTM - 1) / kTM;
  const int64_t n = static_cast<int64_t>(a.n_otiles) * a.n_mtiles;
  if (n > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  if (small_c)
    hipLaunchKernelGGL((fold_conv_kernel<kBits, kNWO, kMB, true>), dim3(static_cast<uint32_t>(n)),
                       dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((fold_conv_kernel<kBits, kNWO, kMB, false>), dim3(static_cast<uint32_t>(n)),
                       dim3(kThreads), 0, st, a);
  return last_launch();
}

// Rows per wave (kMB blocks of 16) are chosen so that the workgroups fill
// the 256 compute units in as few rounds as possible: cost = rounds * kMB.
template <int kBits, int kNWO>
fgq_status launch_nwo(const FoldArgs& a, hipStream_t st) {
  constexpr int kNWM = 4 / kNWO;
  const int64_t otiles = ceil_div(a.O, 32 * kNWO);
  int best = 8;
  int64_t best_cost = -1;
  for (int mb = 8; mb >= 4; --mb) {
    const int64_t tiles = otiles * ceil_div(a.M, kNWM * mb * 16);
    const int64_t cost = ceil_div(tiles, 256) * mb;
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best = mb;
    }
  }
  switch (best) {
    case 4: return launch_cfg<kBits, kNWO, 4>(a, st);
    case 5: return launch_cfg<kBits, kNWO, 5>(a, st);
    case 6: return launch_cfg<kBits, kNWO, 6>(a, st);
    case 7: return launch_cfg<kBits, kNWO, 7>(a, st);
    default: return launch_cfg<kBits, kNWO, 8>(a, st);
  }
}

template <int kBits>
fgq_status launch_bits(const FoldArgs& a, hipStream_t st) {
  if (a.O > 64) return launch_nwo<kBits, 4>(a, st);
  if (a.O > 32) return launch_nwo<kBits, 2>(a, st);
  return launch_nwo<kBits, 1>(a, st);
}

}  // namespace

bool fold_supported(const ConvGeom& g, const uint8_t* q) {
  const uintptr_t qa = reinterpret_cast<uintptr_t>(q);
  const int64_t in_elems = g.B * g.H * g.W * g.C;
  return g.C % 16 == 0 && g.K < (1LL << 17) && qa % (g.bits == 8 ? 16 : 8) == 0 &&
         in_elems < (1LL << 31) && g.M < (1LL << 31) && g.O < (1LL << 24) &&
         g.H * g.W < (1LL << 30);
}

fgq_status launch_fold_conv(const uint8_t* q, const float* sx, const void* prepared,
                            const ConvGeom& g, float* y, hipStream_t st) {
  const PreparedLayout L = prepared_layout(g.O, g.K);
  const char* base = static_cast<const char*>(prepared);
  FoldArgs a;
  a.q = q;
  a.sx = sx;
  a.planes = reinterpret_cast<const int8_t*>(base + L.planes_off);
  a.bias = reinterpret_cast<const int32_t*>(base + L.bias_off);
  a.scale = reinterpret_cast<const float*>(base + L.scale_off);
  a.y = y;
  a.M = static_cast<int32_t>(g.M);
  a.K = static_cast<int32_t>(g.K);
  a.O = static_cast<int32_t>(g.O);
  a.Kp = static_cast<int32_t>(L.Kp);
  a.H = static_cast<int32_t>(g.H);
  a.W = static_cast<int32_t>(g.W);
  a.C = static_cast<int32_t>(g.C);
  a.R = g.R;
  a.S = g.S;
  a.Ho = static_cast<int32_t>(g.Ho);
  a.Wo = static_cast<int32_t>(g.Wo);
  a.sh = g.sh;
  a.sw = g.sw;
  a.ph = g.ph;
  a.pw = g.pw;
  a.n_otiles = a.n_mtiles = 0;
  return g.bits == 8 ? launch_bits<8>(a, st) : launch_bits<4>(a, st);
}

// Direct G%64 matrix-core path: not built yet.
bool group64_supported(const ConvGeom&, const uint8_t*) { return false; }
fgq_status launch_group64_conv(const uint8_t*, const float*, const uint8_t*, const float*,
                               const ConvGeom&, float*, hipStream_t) {
  return FGQ_ERR_UNSUPPORTED;
}

}  // namespace fgq
