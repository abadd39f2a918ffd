// prepare.hip -- per-layer constants of the matrix-core kernels.
//
// Group size 64 (a group is two K slices of the 32x32x32 int8 instruction):
// the per-group kernel takes the ternary weights as 2-bit codes in its
// operand order (expanded to int8 in registers) and alpha transposed to
// [K/64][O32], so that one wave reads the alphas of its 32 channels for one
// group as 128 contiguous bytes.
//
// Other group sizes: the folded-scale kernel.
// y[m][o] = s_x * sum_k q[m][k] * alpha[o][g(k)] * t[o][k] is a dense GEMM
// with real weights.  Putting every alpha of channel o on one grid of step
// h_o (the smallest fp32 value with alpha_max(o) / h_o <= 127*(1+255+255^2)),
// A[o][g] = rint(alpha[o][g] / h_o), and writing A in three balanced base-255
// digits d_j in [-127, 127] gives int8 weights t*d_j, so the layer becomes
// three exact int8 products combined as
//   y = s_x * h_o * sum_j 255^j * (S_j + bias_j[o]),
// S_j = sum_k q'[m][k] * t[o][k] * d_j[o][g(k)] over offset activations
// q' = q - 128 (uint8) and bias_j = 128 * sum_k t*d_j (zero for uint4).
// The only departures from the exact value are the rounding of alpha to the
// grid and the final fp32 combination; the accuracy guard below checks the
// first against kFoldMaxRel per scale.
//
// One block per output channel (channels padded to a multiple of 32 get
// zero planes): max alpha -> h_o, then digits, planes (written in the
// fragment order of the matrix-core kernel) and the per-plane sums.  For G
// a power of two in 4..128 the layout also holds the 2-bit codes and each
// group's three digits in the codes-expanding GEMM's order (xlayout.h;
// digits plane-major, [3][O128 * Kp/64 * xnb]), for GEMMs at small batch.
#include "fgq_internal.h"
#include "xlayout.h"

// Every floating-point expression here is evaluated exactly as written.
#pragma clang fp contract(off)

namespace fgq {

PreparedLayout prepared_layout(int64_t O, int64_t K, int32_t G) {
  PreparedLayout L;
  L.O32 = round_up(O, 32);
  L.Kp = round_up(K, 2 * kFoldKStep);  // whole 128-wide kernel steps; k >= K is zero
  L.nks = L.Kp / kFoldKStep;
  L.planes_off = 0;
  if (G == 64 && K / 64 <= kGroupMaxGroups) {
    L.kind = kPrepGroup;
    L.alpha_off = round_up(L.O32 * L.Kp / 4, 256);
    L.total = round_up(L.alpha_off + 4 * L.nks * L.O32, 256);
    L.bias_off = L.scale_off = L.total;
    L.xcodes_off = L.xacodes_off = L.total;
  } else {
    L.kind = kPrepFold;
    L.bias_off = round_up(3 * L.O32 * L.Kp, 256);
    L.scale_off = round_up(L.bias_off + 12 * O, 256);
    const int64_t xnb = dfpx_acode_bytes(G), O128 = round_up(O, 128);
    L.xcodes_off = round_up(L.scale_off + 4 * O, 256);
    L.xacodes_off = round_up(L.xcodes_off + (xnb > 0 ? O128 * L.Kp / 4 : 0), 256);
    L.total = round_up(L.xacodes_off + 3 * O128 * (L.Kp / 64) * xnb, 256);
    L.alpha_off = L.total;
  }
  return L;
}

namespace {

constexpr int kThreads = 256;
constexpr int64_t kAmax = 127LL * (1 + 255 + 255 * 255);  // 8290687

__device__ inline void digits_of(int64_t A, int d[3]) {
  for (int j = 0; j < 3; ++j) {
    int64_t r = A % 255;  // A >= 0
    if (r > 127) r -= 255;
    d[j] = static_cast<int>(r);
    A = (A - r) / 255;
  }
}

// Byte offset of plane j, channel o, reduction index k in the fragment order.
__device__ inline int64_t frag_offset(int64_t nks, int j, int64_t o, int64_t k) {
  const int64_t tile = o / 32, ks = k / kFoldKStep;
  const int kk = static_cast<int>(k % kFoldKStep);
  const int half = kk / 32, lane = static_cast<int>(o % 32) + 32 * ((kk % 32) / 16);
  return (((tile * nks + ks) * 3 + j) * 2 + half) * 1024 + lane * 16 + (kk % 16);
}

__global__ __launch_bounds__(kThreads) void prepare_kernel(
    const uint8_t* __restrict__ codes, const float* __restrict__ alpha, int64_t O,
    int64_t K, int32_t G, int64_t Kp, int8_t* __restrict__ planes,
    int32_t* __restrict__ bias, float* __restrict__ scale, uint8_t* __restrict__ xcodes,
    int8_t* __restrict__ xdigits, int32_t xnb) {
  __shared__ float redf[kThreads / 64];
  __shared__ double redw[kThreads / 64];
  __shared__ int64_t redi[3][kThreads / 64];
  const int64_t o = blockIdx.x;
  const int64_t nks = Kp / kFoldKStep;
  const int64_t nk = Kp / 128, xplane = round_up(O, 128) * nk * 2 * xnb;  // digit plane stride
  if (o >= O) {  // padding channel of the last 32- (or 128-) channel tile
    if (o < round_up(O, 32))
      for (int64_t k = threadIdx.x; k < Kp; k += kThreads)
        for (int j = 0; j < 3; ++j) planes[frag_offset(nks, j, o, k)] = 0;
    if (xnb > 0) {
      write_xcodes(codes, o, K, Kp, false, xcodes);
      for (int64_t e = threadIdx.x; e < nk * 2 * xnb; e += kThreads) {
        const int64_t ln = xfrag_lane(nk, o, e / (2 * xnb), static_cast<int>((e / xnb) % 2));
        for (int j = 0; j < 3; ++j) xdigits[j * xplane + ln * xnb + e % xnb] = 0;
      }
    }
    return;
  }
  const int64_t ng = K / G;
  const int64_t rb = ceil_div(K, 4);
  const int lane = threadIdx.x % 64, wid = threadIdx.x / 64;

  float amax = 0.0f;
  for (int64_t gi = threadIdx.x; gi < ng; gi += kThreads) amax = fmaxf(amax, alpha[o * ng + gi]);
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  if (lane == 0) redf[wid] = amax;
  __syncthreads();
  amax = redf[0];
  for (int i = 1; i < kThreads / 64; ++i) amax = fmaxf(amax, redf[i]);

  // Grid step h: the smallest fp32 value with amax / h <= kAmax, so that the
  // largest scale uses the whole three-digit range (A = rint(alpha / h)).
  float h = 0.0f;
  if (amax > 0.0f) {
    h = static_cast<float>(static_cast<double>(amax) / static_cast<double>(kAmax));
    if (static_cast<double>(h) * static_cast<double>(kAmax) < static_cast<double>(amax))
      h = nextafterf(h, INFINITY);
  }
  const double hd = h;

  // Accuracy guard: the largest relative error of a group scale on the
  // grid, max_g |A_g h - alpha_g| / alpha_g over the channel's non-zero
  // scales (A_g h and the difference are exact in fp64).  The folded result
  // then differs from the exact one by at most that fraction of
  // s_x * sum_g alpha_g |P_g|, plus the fp32 combination (below
  // kFoldCombineRel of the same magnitude); a channel beyond kFoldMaxRel
  // gets a NaN scale, which the host reports.  A negative or non-finite
  // scale, or a step below the normal fp32 range, fails the channel too.
  double worst = (amax > 0.0f && h < __FLT_MIN__) ? INFINITY : 0.0;
  for (int64_t gi = threadIdx.x; gi < ng; gi += kThreads) {
    const float a = alpha[o * ng + gi];
    if (!(a >= 0.0f) || !(a < INFINITY)) {
      worst = INFINITY;
    } else if (a > 0.0f) {
      const double A = rint(static_cast<double>(a) / hd);
      worst = fmax(worst, fabs(A * hd - static_cast<double>(a)) / static_cast<double>(a));
    }
  }
  for (int off = 32; off > 0; off >>= 1) worst = fmax(worst, __shfl_xor(worst, off));
  if (lane == 0) redw[wid] = worst;
  __syncthreads();
  worst = redw[0];
  for (int i = 1; i < kThreads / 64; ++i) worst = fmax(worst, redw[i]);
  const bool fits = worst <= kFoldMaxRel;
  // the grid code of a scale (0 for a zero scale or a failed channel)
  auto grid_code = [&](float a) -> int64_t {
    return fits && a > 0.0f ? static_cast<int64_t>(rint(static_cast<double>(a) / hd)) : 0;
  };

  if (xnb > 0) {
    write_xcodes(codes, o, K, Kp, true, xcodes);
    for (int64_t e = threadIdx.x; e < nk * 2 * xnb; e += kThreads) {
      const int64_t ks = e / (2 * xnb);
      const int hf = static_cast<int>((e / xnb) % 2), jb = static_cast<int>(e % xnb);
      const int64_t k = xscale_k(ks, hf, jb, G);
      int d[3] = {0, 0, 0};
      if (k < K) digits_of(grid_code(alpha[o * ng + k / G]), d);
      const int64_t ln = xfrag_lane(nk, o, ks, hf);
      for (int j = 0; j < 3; ++j) xdigits[j * xplane + ln * xnb + jb] = static_cast<int8_t>(d[j]);
    }
  }

  int64_t s[3] = {0, 0, 0};
  for (int64_t k = threadIdx.x; k < Kp; k += kThreads) {
    int d[3] = {0, 0, 0};
    int t = 0;
    if (k < K) {
      const uint32_t c = (codes[o * rb + k / 4] >> (2 * (k % 4))) & 3u;
      t = c == 1 ? 1 : (c == 3 ? -1 : 0);
      digits_of(grid_code(alpha[o * ng + k / G]), d);
    }
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const int v = t * d[j];
      planes[frag_offset(nks, j, o, k)] = static_cast<int8_t>(v);
      s[j] += v;
    }
  }
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    int64_t v = s[j];
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if (lane == 0) redi[j][wid] = v;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int j = 0; j < 3; ++j) {
      int64_t v = 0;
      for (int i = 0; i < kThreads / 64; ++i) v += redi[j][i];
      bias[j * O + o] = static_cast<int32_t>(128 * v);
    }
    scale[o] = fits ? h : NAN;
  }
}

// Group kind: one block per channel of the padded channel range.  The
// ternary codes go in the per-group kernel's operand order: lane
// l = o%32 + 32*hf of channel tile o/32 holds, in 128-wide step ks, four
// 32-bit words d = 2*blk + h, word d holding the 16 codes of
// k = 128*ks + 64*blk + 32*h + 16*hf + [0, 16) with the code of k0 + 4i + b
// in byte b at bits 2i (so one wave-wide load of a step is one contiguous
// kilobyte, and a word's four permute selectors are a shift and a mask).
__global__ __launch_bounds__(kThreads) void prepare_group_kernel(
    const uint8_t* __restrict__ codes, const float* __restrict__ alpha, int64_t O,
    int64_t K, int64_t Kp, int64_t O32, uint32_t* __restrict__ gcodes,
    float* __restrict__ alpha_t) {
  const int64_t o = blockIdx.x;
  const int64_t nks = Kp / kFoldKStep, nk = Kp / 128, ng = K / 64, rb = ceil_div(K, 4);
  for (int64_t e = threadIdx.x; e < nk * 8; e += kThreads) {
    const int64_t ks = e / 8;
    const int hf = static_cast<int>((e / 4) % 2), d = static_cast<int>(e % 4);
    const int64_t k0 = 128 * ks + 32 * d + 16 * hf;  // 64*blk + 32*h = 32*d
    uint32_t v = 0;
    for (int j = 0; j < 16; ++j) {
      const int64_t k = k0 + j;
      const uint32_t c = (o < O && k < K) ? (codes[o * rb + k / 4] >> (2 * (k % 4))) & 3u : 0u;
      v |= c << (8 * (j % 4) + 2 * (j / 4));
    }
    gcodes[((o / 32 * nk + ks) * 64 + o % 32 + 32 * hf) * 4 + d] = v;
  }
  for (int64_t gi = threadIdx.x; gi < nks; gi += kThreads)
    alpha_t[gi * O32 + o] = (o < O && gi < ng) ? alpha[o * ng + gi] : 0.0f;
}

}  // namespace

fgq_status launch_prepare(const uint8_t* codes, const float* alpha, int64_t O, int64_t K,
                          int32_t G, void* prepared, hipStream_t st) {
  const PreparedLayout L = prepared_layout(O, K, G);
  char* base = static_cast<char*>(prepared);
  if (L.O32 > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  if (L.kind == kPrepGroup) {
    hipLaunchKernelGGL(prepare_group_kernel, dim3(static_cast<uint32_t>(L.O32)), dim3(kThreads), 0,
                       st, codes, alpha, O, K, L.Kp, L.O32,
                       reinterpret_cast<uint32_t*>(base + L.planes_off),
                       reinterpret_cast<float*>(base + L.alpha_off));
    return last_launch();
  }
  const int32_t xnb = static_cast<int32_t>(dfpx_acode_bytes(G));
  const int64_t nblk = xnb > 0 ? round_up(O, 128) : L.O32;
  hipLaunchKernelGGL(prepare_kernel, dim3(static_cast<uint32_t>(nblk)), dim3(kThreads), 0, st, codes,
                     alpha, O, K, G, L.Kp, reinterpret_cast<int8_t*>(base + L.planes_off),
                     reinterpret_cast<int32_t*>(base + L.bias_off),
                     reinterpret_cast<float*>(base + L.scale_off),
                     reinterpret_cast<uint8_t*>(base + L.xcodes_off),
                     reinterpret_cast<int8_t*>(base + L.xacodes_off), xnb);
  return last_launch();
}

}  // namespace fgq
