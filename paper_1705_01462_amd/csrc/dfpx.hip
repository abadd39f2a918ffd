// dfpx.hip -- the GEMM with fixed-point group scales (Sec. 4) for few rows
// and long K (fully-connected layers at small batch), reading the weights
// as stored: 2-bit codes and one int8 scale code A per group, expanded to
// the int8 weights A*t in registers instead of the one-byte-per-weight
// plane of the prepared layout (0.25 + 1/G bytes per weight).
//
// Work split: a workgroup owns 128 channels, kNB 32-row blocks and up to
// kSteps 128-wide K steps (split K: int32 sums per split, reduced by
// splitk_reduce_kernel with the fixed-point epilogue).  Its waves are,
// with two 32-row blocks, two sets of four (a wave per 32 channels), each
// set taking half of the steps, so that two waves share every SIMD and one's
// code expansion overlaps the other's matrix instructions (the sets' sums
// meet in LDS); with one block, one set of four.  Its
// activation slice (kNB*32 rows x kSteps*128 k) is loaded once and stays in
// LDS, and every code and scale-code load of the split is issued up front,
// after the activation loads: the memory counter completes in order, so the
// publish of the slice waits for the activations only, and step s then
// waits for its own weights only.  Nothing in the K loop waits for a later
// load, so the whole split's traffic is in flight at once.
//
// Operand order.  Lane l (channel 32*wave + l%32, half hf = l/32) holds, in
// step s and K quarter h, the 16 weights k = 128*s + 64*hf + 16*h + [0, 16);
// the activation fragment of the same lane reads the same 16 k of its row
// from LDS.  The prepared layout stores the codes and the scale codes in
// exactly this order ([O/128][K/128][4 waves][64 lanes][16 code bytes, or
// 64/G scale-code bytes]), so every weight load of a wave reads one
// contiguous block (a kilobyte of codes), and within a quarter's 32 bits of
// codes byte b holds, at bits 2i, the code of weight 4i+b: the codes of
// weights 4i..4i+3 are the bytes of (codes >> 2i) & 0x03030303.
//
// Expansion (xexpand.h): each weight's code is turned into a byte selector
// by a permute through a constant table, then one permute per four weights
// picks 0, A or -A from the scale bytes and their negations.  Code 2 is
// never written.
//
// Padding: codes and scale codes past K and past O are zero in the prepared
// layout, so padded activations (past K, or rows past M) meet zero weights;
// the uint8 offset term covers k < K only, as the 128 * sum of the weights
// in the prepared bias.  Partial sums go out through LDS as 16-byte row
// pieces when O % 4 == 0 and the workspace is 16-byte aligned.
#include <algorithm>

#include "fgq_internal.h"
#include "igemm.h"
#include "xexpand.h"

namespace fgq {
namespace {

using namespace ig;

constexpr int kSteps = 8;  // K steps per split at most (LDS: kNB * 32 KB)

struct DfpxArgs {
  const uint8_t* q;       // activations [M][K] (uint8) or [M][K/2] (uint4)
  const uint8_t* xcodes;  // codes, expanding-GEMM order
  const int8_t* xacodes;  // per plane: scale codes (or scale digits), same order
  const int32_t* bias;    // [planes][O]  128 * sum_k (weight of the plane) (uint8 offset term)
  int32_t* part;          // [splits][planes][M][O]
  int32_t M, K, O, n_otiles, n_mtiles, splits, sps, nk, staged;
  int32_t q_bytes, xcodes_bytes, xacodes_bytes, xplane;  // xplane: bytes between planes
};

template <int kNB, int kPlanes>
constexpr int wg_threads() { return kNB == 2 || kPlanes == 3 ? 512 : 256; }

template <int kBits, int kG, int kNB, int kPlanes>
__global__ __launch_bounds__((wg_threads<kNB, kPlanes>()), 2) void dfpx_gemm_kernel(DfpxArgs a) {
  constexpr int kWG = wg_threads<kNB, kPlanes>();
  constexpr int kSets = kWG / 256;                    // wave sets sharing the steps
  constexpr int kRows = 32 * kNB;
  constexpr int kStageB = kRows * kRowB;              // one step's activations
  constexpr int kXP = kRows * kSteps * kSlots / kWG;  // 16-k pieces per thread
  constexpr int kHalf = kSteps / kSets;               // steps per wave
  __shared__ __attribute__((aligned(16))) unsigned char lds[kSteps * kStageB];

  const int tid = threadIdx.x;
  const int lane = tid % 64, wo = (tid / 64) % 4, sh = tid / 256, hf = lane / 32;
  const int ntiles = a.n_otiles * a.n_mtiles;
  const int tsplit = xcd_swizzle(blockIdx.x, ntiles * a.splits);
  const int split = tsplit / ntiles, tile = tsplit % ntiles;
  const int oc = (tile % a.n_otiles) * 128 + 32 * wo + lane % 32;  // the lane's channel
  const int m0 = (tile / a.n_otiles) * kRows;
  const int nk_all = (a.K + kKT - 1) / kKT;
  const int ks0 = split * a.sps;
  const int nsteps = ks0 + a.sps < nk_all ? a.sps : nk_all - ks0;  // 1..kSteps
  const int k0 = ks0 * kKT;

  // The uint8 offset term of the lane's channel (split 0, first half only),
  // requested first so that no wait for it follows the weight loads.
  const bool ocok = oc < a.O;
  int bj[kPlanes] = {};
  if constexpr (kBits == 8) {
    const Buf brs = make_buf(a.bias, 4 * kPlanes * a.O, kSiteBias, kBufFlags);
#pragma unroll
    for (int j = 0; j < kPlanes; ++j)
      bj[j] = static_cast<int>(buf_load_b32(brs, ocok && ks0 == 0 && sh == 0 ? 4 * (j * a.O + oc) : kOutOfRange, 0));
  }

  // ---- activation slice: piece p = tid + 512*i is row p / (8*kSteps),
  // 16-k slot p % (8*kSteps) (a row's slots are consecutive threads, so a
  // wave reads one contiguous kilobyte of a row).  Rows >= M and steps past
  // the split read nothing.
  const Buf qrs = make_buf(a.q, a.q_bytes, kSiteActs, kBufFlags);
  typedef typename std::conditional<kBits == 8, v4i, v2i>::type raw_t;
  raw_t xraw[kXP];
#pragma unroll
  for (int i = 0; i < kXP; ++i) {
    const int p = tid + kWG * i;
    const int row = p / (kSlots * kSteps), ksl = p % (kSlots * kSteps);
    const int m = m0 + row, k = k0 + 16 * ksl;
    const bool ok = (m < a.M) & (ksl < kSlots * nsteps) & (k < a.K);
    const uint32_t e = static_cast<uint32_t>(m) * static_cast<uint32_t>(a.K) + static_cast<uint32_t>(k);
    if constexpr (kBits == 8)
      xraw[i] = buf_load_b128(qrs, ok ? e : kOutOfRange, 0);
    else
      xraw[i] = buf_load_b64(qrs, ok ? e >> 1 : kOutOfRange, 0);
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- every weight load of the wave's steps (kHalf*sh + s), in the
  // prepared order.  Steps past the split re-read the split's last step (in
  // range; never used).
  const Buf crs = make_buf(a.xcodes, a.xcodes_bytes, kSiteCodes, kBufFlags);
  const Buf ars = make_buf(a.xacodes, a.xacodes_bytes, kSiteScales, kBufFlags);
  const int lane0 = ((tile % a.n_otiles) * a.nk + ks0) * 256 + 64 * wo + lane;  // lane index of step ks0
  constexpr int kAB = ACodes<kG>::kBytes;
  v4i cw[kHalf];
  ACodes<kG> aw[kPlanes][kHalf];
#pragma unroll
  for (int s = 0; s < kHalf; ++s) {
    const int st = kHalf * sh + s;
    const int ln = lane0 + 256 * (st < nsteps ? st : nsteps - 1);
    cw[s] = buf_load_b128(crs, 16 * ln, 0);
#pragma unroll
    for (int j = 0; j < kPlanes; ++j) aw[j][s].load(ars, j * a.xplane + kAB * ln);
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- publish the slice: uint8 as q - 128, uint4 unpacked
#pragma unroll
  for (int i = 0; i < kXP; ++i) {
    const int p = tid + kWG * i;
    const int row = p / (kSlots * kSteps), ksl = p % (kSlots * kSteps);
    unsigned char* dst = lds + (ksl / kSlots) * kStageB + lds_off(row, ksl % kSlots);
    v4i v;
    if constexpr (kBits == 8) {
      const int x = static_cast<int>(0x80808080u);
      v = xraw[i];
      v.x ^= x; v.y ^= x; v.z ^= x; v.w ^= x;
    } else {
      v = unpack_u4x16(static_cast<uint32_t>(xraw[i].x), static_cast<uint32_t>(xraw[i].y));
    }
    *reinterpret_cast<v4i*>(dst) = v;
  }
  __syncthreads();

  v16i acc[kPlanes][kNB];
#pragma unroll
  for (int j = 0; j < kPlanes; ++j)
#pragma unroll
    for (int c = 0; c < kNB; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][c][r] = bj[j];
  int afrag[kNB][4];
#pragma unroll
  for (int c = 0; c < kNB; ++c)
#pragma unroll
    for (int h = 0; h < 4; ++h) afrag[c][h] = lds_off(32 * c + lane % 32, 4 * hf + h);

#pragma unroll
  for (int s = 0; s < kHalf; ++s) {
    const int st = kHalf * sh + s;
    if (st >= nsteps) break;
    const unsigned char* base = lds + st * kStageB;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      uint32_t sel[4];
      selectors<kG>(static_cast<uint32_t>(cw[s][h]), sel);
      v4i xf[kNB];
#pragma unroll
      for (int c = 0; c < kNB; ++c) xf[c] = *reinterpret_cast<const v4i*>(base + afrag[c][h]);
#pragma unroll
      for (int j = 0; j < kPlanes; ++j) {
        const v4i wf = expand16(sel, aw[j][s].quarter(h));
#pragma unroll
        for (int c = 0; c < kNB; ++c) acc[j][c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xf[c], wf, acc[j][c], 0, 0, 0);
      }
    }
  }

  // ---- the sums into a kRows x 128-channel int32 tile in LDS (the slice
  // is dead once every wave is past the K loop); a second wave set adds its
  // own with LDS atomic adds (integer, so the order does not matter)
  constexpr int kPitch = 128 * 4 + 32;  // the two rows of a write are 32 banks apart
  static_assert(kRows * kPitch <= kSteps * kStageB, "partial tile fits the slice");
  auto at = [&](int c, int r) -> int* {
    const int row = 32 * c + 8 * (r / 4) + 4 * hf + (r % 4);
    return reinterpret_cast<int*>(lds + row * kPitch + 4 * (32 * wo + lane % 32));
  };
#pragma unroll
  for (int j = 0; j < kPlanes; ++j) {
    int32_t* const part = a.part + (static_cast<int64_t>(split) * kPlanes + j) * a.M * a.O;
    // element range of this split's plane j (checking builds)
    const int64_t pbase = (static_cast<int64_t>(split) * kPlanes + j) * a.M * a.O;
    const int64_t plimit = static_cast<int64_t>(a.splits) * kPlanes * a.M * a.O;
    if (kSets == 1 && !a.staged) {
      if (ocok) {
#pragma unroll
        for (int c = 0; c < kNB; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int m = m0 + 32 * c + 8 * (r / 4) + 4 * hf + (r % 4);
            const int64_t e = static_cast<int64_t>(m) * a.O + oc;
            if (m < a.M && check_store(kSiteStorePart, pbase + e, 1, plimit)) part[e] = acc[j][c][r];
          }
      }
      continue;
    }
    __syncthreads();  // the slice (or the previous plane's tile) is no longer read
    if (sh == 0) {
#pragma unroll
      for (int c = 0; c < kNB; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) *at(c, r) = acc[j][c][r];
    }
    if constexpr (kSets == 2) {
      __syncthreads();
      if (sh == 1) {
#pragma unroll
        for (int c = 0; c < kNB; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            __hip_atomic_fetch_add(at(c, r), acc[j][c][r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
      if (!a.staged) {
        __syncthreads();
        if (sh == 0 && ocok) {
#pragma unroll
          for (int c = 0; c < kNB; ++c)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int m = m0 + 32 * c + 8 * (r / 4) + 4 * hf + (r % 4);
              const int64_t e = static_cast<int64_t>(m) * a.O + oc;
              if (m < a.M && check_store(kSiteStorePart, pbase + e, 1, plimit)) part[e] = *at(c, r);
            }
        }
        continue;
      }
    }
    // this split's raw sums of plane j, [split][j][m][o], as 16-byte pieces of rows
    __syncthreads();
    const int o0 = (tile % a.n_otiles) * 128;
#pragma unroll
    for (int t = tid; t < kRows * 32; t += kWG) {
      const int row = t / 32, ch = o0 + 4 * (t % 32);
      const int m = m0 + row;
      const int64_t e = static_cast<int64_t>(m) * a.O + ch;
      if (m < a.M && ch < a.O && check_store(kSiteStorePart, pbase + e, 4, plimit))
        *reinterpret_cast<v4i*>(part + e) = *reinterpret_cast<const v4i*>(lds + row * kPitch + 16 * (t % 32));
    }
  }
}

template <int kBits, int kNB, int kPlanes>
fgq_status launch_g(const DfpxArgs& a, int G, hipStream_t st) {
  const dim3 grid(static_cast<uint32_t>(a.n_otiles * a.n_mtiles * a.splits));
  constexpr int kWG = wg_threads<kNB, kPlanes>();
  switch (G) {
    case 4: hipLaunchKernelGGL((dfpx_gemm_kernel<kBits, 4, kNB, kPlanes>), grid, dim3(kWG), 0, st, a); break;
    case 8: hipLaunchKernelGGL((dfpx_gemm_kernel<kBits, 8, kNB, kPlanes>), grid, dim3(kWG), 0, st, a); break;
    case 16: hipLaunchKernelGGL((dfpx_gemm_kernel<kBits, 16, kNB, kPlanes>), grid, dim3(kWG), 0, st, a); break;
    case 32: hipLaunchKernelGGL((dfpx_gemm_kernel<kBits, 32, kNB, kPlanes>), grid, dim3(kWG), 0, st, a); break;
    case 64: hipLaunchKernelGGL((dfpx_gemm_kernel<kBits, 64, kNB, kPlanes>), grid, dim3(kWG), 0, st, a); break;
    default: hipLaunchKernelGGL((dfpx_gemm_kernel<kBits, 128, kNB, kPlanes>), grid, dim3(kWG), 0, st, a); break;
  }
  return last_launch();
}

template <int kPlanes>
fgq_status launch_planes(const DfpxArgs& a, int bits, int nb, int G, hipStream_t st) {
  return bits == 8 ? (nb == 1 ? launch_g<8, 1, kPlanes>(a, G, st) : launch_g<8, 2, kPlanes>(a, G, st))
                   : (nb == 1 ? launch_g<4, 1, kPlanes>(a, G, st) : launch_g<4, 2, kPlanes>(a, G, st));
}

// Arguments shared by the two layouts; the caller fills in the pointers.
DfpxArgs make_args(const uint8_t* q, const ConvGeom& g, int32_t* ws, int nb) {
  DfpxArgs a;
  a.q = q;
  a.part = ws;
  a.M = static_cast<int32_t>(g.M);
  a.K = static_cast<int32_t>(g.K);
  a.O = static_cast<int32_t>(g.O);
  a.n_otiles = static_cast<int32_t>(ceil_div(g.O, 128));
  a.n_mtiles = static_cast<int32_t>(ceil_div(g.M, 32 * nb));
  a.splits = dfpx_splits(g.M, g.K, g.O, g.G, &a.sps);
  a.nk = static_cast<int32_t>(round_up(g.K, 128) / 128);
  a.staged = g.O % 4 == 0 && reinterpret_cast<uintptr_t>(ws) % 16 == 0;
  a.q_bytes = static_cast<int32_t>(g.bits == 8 ? g.M * g.K : g.M * g.K / 2);
  return a;
}

}  // namespace

bool dfpx_shape_ok(int64_t M, int64_t K, int64_t O, int32_t G) {
  const int64_t O128 = round_up(O, 128), Kp = round_up(K, 128);
  return dfpx_acode_bytes(G) > 0 && M <= kDfpxMaxM && K % 16 == 0 && K <= kFoldMaxK &&
         O128 * Kp / 4 < (1LL << 31) && M * K < (1LL << 31) && M * O < (1LL << 31);
}

bool dfpx_supported(const ConvGeom& g, const uint8_t* q) {
  const uintptr_t align = g.bits == 8 ? 16 : 8;
  // a 1x1 convolution at stride 1 without padding is the GEMM on [M][K]
  return g.R == 1 && g.S == 1 && g.sh == 1 && g.sw == 1 && g.ph == 0 && g.pw == 0 &&
         reinterpret_cast<uintptr_t>(q) % align == 0 && dfpx_shape_ok(g.M, g.K, g.O, g.G);
}

int32_t dfpx_splits(int64_t M, int64_t K, int64_t O, int32_t G, int32_t* steps_per_split) {
  (void)M;
  (void)O;
  (void)G;
  // As many steps per split as the LDS slice holds: a workgroup's loads are
  // all in flight at once, so its time is about one memory round trip plus
  // its bytes, and fewer splits mean fewer int32 sums to write and reduce.
  const int64_t nk = ceil_div(K, 128);
  const int64_t splits = ceil_div(nk, kSteps);
  const int64_t sps = ceil_div(nk, splits);
  *steps_per_split = static_cast<int32_t>(sps);
  return static_cast<int32_t>(ceil_div(nk, sps));
}

fgq_status launch_dfpx_splitk(const uint8_t* q, const float* sx, const void* prepared,
                              const ConvGeom& g, const LayerOut& out, int32_t* ws, hipStream_t st) {
  const PreparedLayout L = prepared_layout_dfp(g.O, g.K, g.G);
  const char* base = static_cast<const char*>(prepared);
  const int nb = g.M <= 32 ? 1 : 2;
  DfpxArgs a = make_args(q, g, ws, nb);
  a.xcodes = reinterpret_cast<const uint8_t*>(base + L.xcodes_off);
  a.xacodes = reinterpret_cast<const int8_t*>(base + L.xacodes_off);
  a.bias = reinterpret_cast<const int32_t*>(base + L.bias_off);
  a.xcodes_bytes = static_cast<int32_t>(L.xacodes_off - L.xcodes_off);
  a.xacodes_bytes = static_cast<int32_t>(L.total - L.xacodes_off);
  a.xplane = 0;
  if (static_cast<int64_t>(a.n_otiles) * a.n_mtiles * a.splits > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  fgq_status rc = launch_planes<1>(a, g.bits, nb, g.G, st);
  if (rc != FGQ_OK) return rc;
  return launch_splitk_reduce(ws, a.splits, /*dfp=*/true, g.M, g.O, sx, nullptr,
                              reinterpret_cast<const int32_t*>(base), out, st);
}

fgq_status launch_foldx_splitk(const uint8_t* q, const float* sx, const void* prepared,
                               const ConvGeom& g, const LayerOut& out, int32_t* ws, hipStream_t st) {
  const PreparedLayout L = prepared_layout(g.O, g.K, g.G);
  const char* base = static_cast<const char*>(prepared);
  const int nb = g.M <= 32 ? 1 : 2;
  DfpxArgs a = make_args(q, g, ws, nb);
  a.xcodes = reinterpret_cast<const uint8_t*>(base + L.xcodes_off);
  a.xacodes = reinterpret_cast<const int8_t*>(base + L.xacodes_off);
  a.bias = reinterpret_cast<const int32_t*>(base + L.bias_off);
  a.xcodes_bytes = static_cast<int32_t>(L.xacodes_off - L.xcodes_off);
  a.xacodes_bytes = static_cast<int32_t>(L.total - L.xacodes_off);
  a.xplane = static_cast<int32_t>(round_up(g.O, 128) * (L.Kp / 64) * dfpx_acode_bytes(g.G));
  if (static_cast<int64_t>(a.n_otiles) * a.n_mtiles * a.splits > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  fgq_status rc = launch_planes<3>(a, g.bits, nb, g.G, st);
  if (rc != FGQ_OK) return rc;
  return launch_splitk_reduce(ws, a.splits, /*dfp=*/false, g.M, g.O, sx,
                              reinterpret_cast<const float*>(base + L.scale_off), nullptr, out, st);
}

}  // namespace fgq
