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
// channels and walks K in steps of 128 (four 32-wide K slices of the
// v_mfma_i32_32x32x32_i8 instruction, which runs at twice the rate of the
// 16x16x64 form on gfx950; the prepared K is padded to a multiple of 128
// with zero weights).  Its four waves are kNWO (channels) x 4/kNWO
// (rows); each wave owns 32 channels x kNB*32 rows, i.e. kNB 32x32 blocks
// per digit plane.
//  * Activations are the 32-row MFMA operand: gathered into LDS once per
//    workgroup per step (double-buffered, 128-byte rows with the 16-byte
//    slot XOR-swizzled by (row/2) % 8 so that both the row writes and the
//    32-row fragment reads hit every bank once per pass) and read by every
//    wave that shares those rows.
//  * Weights are the 32-column operand: raw buffer loads straight into
//    registers (every workgroup reads the same few hundred KB, so they come
//    from L2).  They are stored in fragment order, so each wave-wide load is
//    one contiguous kilobyte; a lane's offset is fixed and the K step is the
//    scalar offset, so the loop spends no vector instructions on them.
//  * Out-of-image activation pieces are loaded with an offset past the
//    buffer end, which the hardware returns as zeros (q = 0, then q' = -128
//    for uint8), so padding needs no select.
// The accumulators start at the per-plane bias (uint8), and the loads of
// step ks+1 are interleaved between the matrix instructions of step ks.
// A lane's 16 accumulators of a block are 16 rows of one channel; for each
// row the wave stores 32 consecutive channels (128 contiguous bytes).
// Workgroups are numbered so that consecutive row tiles land on one XCD
// (shared halos in that XCD's L2).  In-loop index arithmetic is 32-bit and
// incremental.
#include <type_traits>

#include "fgq_internal.h"

namespace fgq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef int v2i __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kKT = 128;     // K per step (two fragment-ordered 64-wide blocks)
constexpr int kRowB = kKT;   // LDS bytes per activation row (one step of K)
constexpr int kSlots = kKT / 16;  // 16-byte k-slots per row
constexpr int kBufFlags = 0x00020000;  // raw buffer descriptor word 3 (gfx9)
constexpr uint32_t kOutOfRange = 0x80000000u;

struct FoldArgs {
  const uint8_t* q;
  const float* sx;
  const int8_t* planes;
  const int32_t* bias;
  const float* scale;
  float* y;
  int32_t M, K, O, nks;
  int32_t H, W, C, R, S, Ho, Wo, sh, sw, ph, pw;
  int32_t q_bytes, planes_bytes;
  int32_t n_otiles, n_mtiles;
};

// Unpack 16 four-bit values (8 bytes, element 2i in the low nibble) to 16
// bytes in element order.
__device__ inline v4i unpack_u4x16(uint32_t x0, uint32_t x1) {
  const uint32_t lo0 = x0 & 0x0F0F0F0Fu, hi0 = (x0 >> 4) & 0x0F0F0F0Fu;
  const uint32_t lo1 = x1 & 0x0F0F0F0Fu, hi1 = (x1 >> 4) & 0x0F0F0F0Fu;
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

// Byte offset of the 16-byte k-slot `slot` of activation row `row` in LDS.
// The slot is XOR-swizzled by row/2 so that 16 consecutive rows at one slot
// (a fragment read) and 2 rows x 8 slots (a publish) each cover all 64
// banks once.
__device__ inline int lds_off(int row, int slot) {
  return row * kRowB + 16 * (slot ^ ((row >> 1) & (kSlots - 1)));
}

template <int kBits, int kNWO, int kNB, bool kSmallC>
__global__ __launch_bounds__(kThreads, 1) void fold_conv_kernel(FoldArgs a) {
  constexpr int kNWM = 4 / kNWO;
  constexpr int kTO = 32 * kNWO;
  constexpr int kTM = kNWM * kNB * 32;
  constexpr int kPieces = kTM * kSlots;  // 16-element pieces of one activation step
  constexpr int kXP = (kPieces + kThreads - 1) / kThreads;
  // Pieces past the tile (when kTM*4 is not a multiple of 256) go to spare
  // rows after the tile so that every store is unconditional.
  constexpr int kStage = (kTM + (kXP * kThreads - kPieces) / kSlots) * kRowB;
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * kStage];

  const int tid = threadIdx.x;
  const int lane = tid % 64, wave = tid / 64;
  const int wo = wave % kNWO, wm = wave / kNWO;
  const int tile = xcd_swizzle(blockIdx.x, a.n_otiles * a.n_mtiles);
  const int o0 = (tile % a.n_otiles) * kTO + 32 * wo;  // this wave's first channel
  const int m0 = (tile / a.n_otiles) * kTM;             // workgroup's first row

  const __amdgpu_buffer_rsrc_t qrs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(a.q), 0, a.q_bytes, kBufFlags);
  const __amdgpu_buffer_rsrc_t wrs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(a.planes), 0, a.planes_bytes, kBufFlags);

  // ---- weight fragments: lane supplies channel o0 + lane%32, k-slot
  // 16*(lane/32) of K half h; the fragment-ordered planes put the wave's
  // 64 lanes x 16 bytes of (tile, step, plane, half) in one kilobyte.
  const int wbase = (o0 / 32) * a.nks * static_cast<int>(kFoldTileBytes) + 16 * lane;

  // ---- activation pieces owned by this thread: piece p = tid + 256*i is
  // row p/kSlots of the tile, k-slot 16*(p%kSlots) = 16*(tid%kSlots) of each
  // step.
  const int sub = tid % kSlots;
  int rowbase[kXP], hi0[kXP], wi0[kXP];
  bool rowok[kXP];
#pragma unroll
  for (int i = 0; i < kXP; ++i) {
    const int p = tid + kThreads * i;
    const int m = m0 + p / kSlots;
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
  int xlds[kXP];
#pragma unroll
  for (int i = 0; i < kXP; ++i) {
    const int p = tid + kThreads * i;
    xlds[i] = lds_off(p / kSlots, p % kSlots);
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
    if constexpr (kSmallC) {  // C < 128: several taps per step
      const int t = ts + (tc + kKT) / a.C;
      tc = (tc + kKT) % a.C;
      tr += t / a.S;
      ts = t % a.S;
    } else {                  // C >= 128: at most one tap boundary per step
      tc += kKT;
      const bool wrap = tc >= a.C;
      tc = wrap ? tc - a.C : tc;
      const int t = ts + (wrap ? 1 : 0);
      const bool wrap2 = t == a.S;
      ts = wrap2 ? 0 : t;
      tr += wrap2 ? 1 : 0;
    }
  };

  typedef typename std::conditional<kBits == 8, v4i, v2i>::type raw_t;
  raw_t xraw[kXP];
  auto load_x = [&]() {
#pragma unroll
    for (int i = 0; i < kXP; ++i) {
      // Branch-free bounds test (bitwise, no short-circuit) so that the
      // whole step stays one basic block for the scheduler.
      const int hi = hi0[i] + tr, wi = wi0[i] + ts;
      const bool ok = rowok[i] & (tk < a.K) & (static_cast<unsigned>(hi) < static_cast<unsigned>(a.H)) &
                      (static_cast<unsigned>(wi) < static_cast<unsigned>(a.W));
      const int e = (rowbase[i] + tr * a.W + ts) * a.C + tc;  // element offset
      if constexpr (kBits == 8) {
        const uint32_t off = ok ? static_cast<uint32_t>(e) : kOutOfRange;
        xraw[i] = __builtin_amdgcn_raw_buffer_load_b128(qrs, off, 0, 0);
      } else {
        const uint32_t off = ok ? static_cast<uint32_t>(e) >> 1 : kOutOfRange;
        xraw[i] = __builtin_amdgcn_raw_buffer_load_b64(qrs, off, 0, 0);
      }
    }
  };
  auto store_x = [&](int stage) {
    unsigned char* base = lds + stage * kStage;
#pragma unroll
    for (int i = 0; i < kXP; ++i) {
      v4i v;
      if constexpr (kBits == 8) {
        const int x = static_cast<int>(0x80808080u);
        v = xraw[i];
        v.x ^= x; v.y ^= x; v.z ^= x; v.w ^= x;  // q - 128 (padding read 0 -> -128)
      } else {
        v = unpack_u4x16(static_cast<uint32_t>(xraw[i].x), static_cast<uint32_t>(xraw[i].y));
      }
      *reinterpret_cast<v4i*>(base + xlds[i]) = v;
    }
  };

  // A step covers two 64-wide fragment blocks (K quarters hq = 2*blk + h).
  // Loads past the last block read zeros or another tile's weights; they
  // are never used.
  v4i wring[2][3][4];
  auto load_w = [&](auto U, int ks) {
    constexpr int u = decltype(U)::value;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      const int kso = (2 * ks + blk) * static_cast<int>(kFoldTileBytes);
#pragma unroll
      for (int j = 0; j < 3; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          wring[u][j][2 * blk + h] =
              __builtin_amdgcn_raw_buffer_load_b128(wrs, wbase + (2 * j + h) * 1024, kso, 0);
    }
  };

  // Accumulators start at the uint8 offset term 128 * sum_k plane_j[o][k]
  // of the lane's channel, so the epilogue needs no integer additions.
  v16i acc[3][kNB];
  {
    const int oc = o0 + lane % 32;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const int bj = (kBits == 8 && oc < a.O) ? a.bias[j * a.O + oc] : 0;
      v16i init;
#pragma unroll
      for (int r = 0; r < 16; ++r) init[r] = bj;
#pragma unroll
      for (int c = 0; c < kNB; ++c) acc[j][c] = init;
    }
  }

  // A-operand fragment addresses (row = wave rows + 32c + lane%32, slot
  // 2*quarter + lane/32)
  int afrag[kNB][4];
#pragma unroll
  for (int c = 0; c < kNB; ++c)
#pragma unroll
    for (int h = 0; h < 4; ++h) afrag[c][h] = lds_off(wm * kNB * 32 + 32 * c + lane % 32, 2 * h + lane / 32);

  auto compute = [&](int stage, const v4i (&w)[3][4]) {
    const unsigned char* base = lds + stage * kStage;
    v4i xf[kNB][4];
#pragma unroll
    for (int c = 0; c < kNB; ++c)
#pragma unroll
      for (int h = 0; h < 4; ++h) xf[c][h] = *reinterpret_cast<const v4i*>(base + afrag[c][h]);
#pragma unroll
    for (int h = 0; h < 4; ++h)
#pragma unroll
      for (int c = 0; c < kNB; ++c)
#pragma unroll
        for (int j = 0; j < 3; ++j)
          acc[j][c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xf[c][h], w[j][h], acc[j][c], 0, 0, 0);
  };

  // Step ks: prefetch step ks+1 (weights into ring slot (ks+1)%2,
  // activations into registers), feed the matrix cores from LDS stage ks%2
  // and ring slot ks%2, then publish the prefetched activations to the
  // other LDS stage.  Loads past the last step are clamped (weights) or
  // read nothing (activations), so the step has no data-dependent branch;
  // the loop is unrolled by 2 so that ring indices are constants.
  const int nk = (a.K + kKT - 1) / kKT;
  auto step = [&](auto U, int ks) {
    constexpr int u = decltype(U)::value;
    load_w(std::integral_constant<int, 1 - u>{}, ks + 1);
    advance_tap();
    load_x();
    compute(u, wring[u]);
    // Schedule: every fragment read first (distinct registers, LDS latency
    // paid once), then the matrix instructions with the prefetch loads and
    // their address arithmetic slotted between them, so the per-CU load
    // path works while the matrix cores do.
#pragma unroll
    for (int i = 0; i < 4 * kNB; ++i) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
    for (int i = 0; i < 12 + kXP; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 12 * kNB - 2 * (12 + kXP) > 0 ? 12 * kNB - 2 * (12 + kXP) : 0, 0);
    __builtin_amdgcn_sched_barrier(0);  // the publish waits for the prefetch: keep it last
    store_x(1 - u);
    __syncthreads();
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  load_w(I0{}, 0);
  load_x();
  store_x(0);
  __syncthreads();
  int ks = 0;
  for (; ks + 2 <= nk; ks += 2) {
    step(I0{}, ks);
    step(I1{}, ks + 1);
  }
  if (ks < nk) step(I0{}, ks);

  // ---- epilogue: lane holds rows m of channel o.
  const int o = o0 + lane % 32;
  if (o >= a.O) return;
  const float sx = *a.sx;
  const float c0 = sx * a.scale[o];
  const float c1 = c0 * 255.0f, c2 = c0 * 65025.0f;
#pragma unroll
  for (int c = 0; c < kNB; ++c) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * kNB * 32 + 32 * c + 8 * (r / 4) + 4 * (lane / 32) + (r % 4);
      if (m >= a.M) continue;
      const float f2 = static_cast<float>(acc[2][c][r]);
      const float f1 = static_cast<float>(acc[1][c][r]);
      const float f0 = static_cast<float>(acc[0][c][r]);
      __builtin_nontemporal_store(fmaf(f2, c2, fmaf(f1, c1, f0 * c0)),
                                  a.y + static_cast<int64_t>(m) * a.O + o);
    }
  }
}

template <int kBits, int kNWO, int kNB>
fgq_status launch_cfg(const FoldArgs& a0, hipStream_t st) {
  constexpr int kTO = 32 * kNWO, kTM = (4 / kNWO) * kNB * 32;
  FoldArgs a = a0;
  a.n_otiles = (a.O + kTO - 1) / kTO;
  a.n_mtiles = (a.M + kTM - 1) / kTM;
  const int64_t n = static_cast<int64_t>(a.n_otiles) * a.n_mtiles;
  if (n > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  if (a.C < kKT)
    hipLaunchKernelGGL((fold_conv_kernel<kBits, kNWO, kNB, true>), dim3(static_cast<uint32_t>(n)),
                       dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((fold_conv_kernel<kBits, kNWO, kNB, false>), dim3(static_cast<uint32_t>(n)),
                       dim3(kThreads), 0, st, a);
  return last_launch();
}

// Rows per wave (kNB blocks of 32) are chosen so that the workgroups fill
// the 256 compute units in as few rounds as possible: cost = rounds * kNB.
template <int kBits, int kNWO>
fgq_status launch_nwo(const FoldArgs& a, hipStream_t st) {
  constexpr int kNWM = 4 / kNWO;
  const int64_t otiles = ceil_div(a.O, 32 * kNWO);
  int best = 4;
  int64_t best_cost = -1;
  for (int nb = 4; nb >= 2; --nb) {
    const int64_t tiles = otiles * ceil_div(a.M, kNWM * nb * 32);
    const int64_t cost = ceil_div(tiles, 256) * nb;
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
fgq_status launch_bits(const FoldArgs& a, hipStream_t st) {
  if (a.O > 64) return launch_nwo<kBits, 4>(a, st);
  if (a.O > 32) return launch_nwo<kBits, 2>(a, st);
  return launch_nwo<kBits, 1>(a, st);
}

}  // namespace

bool fold_supported(const ConvGeom& g, const uint8_t* q) {
  const uintptr_t qa = reinterpret_cast<uintptr_t>(q);
  const int64_t in_elems = g.B * g.H * g.W * g.C;
  const PreparedLayout L = prepared_layout(g.O, g.K);
  const int64_t plane_bytes = 3 * L.O32 * L.Kp;
  return g.C % 16 == 0 && g.K < (1LL << 17) && qa % (g.bits == 8 ? 16 : 8) == 0 &&
         in_elems < (1LL << 31) && g.M < (1LL << 31) && plane_bytes < (1LL << 31);
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
  a.nks = static_cast<int32_t>(L.nks);
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
  const int64_t in_elems = g.B * g.H * g.W * g.C;
  a.q_bytes = static_cast<int32_t>(g.bits == 8 ? in_elems : in_elems / 2);
  a.planes_bytes = static_cast<int32_t>(3 * L.O32 * L.Kp);
  a.n_otiles = a.n_mtiles = 0;
  return g.bits == 8 ? launch_bits<8>(a, st) : launch_bits<4>(a, st);
}

}  // namespace fgq
