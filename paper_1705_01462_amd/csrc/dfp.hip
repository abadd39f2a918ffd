// dfp.hip -- fixed-point group scales (Sec. 4: the scaling factors are
// quantized to an 8- or 4-bit fixed point) and the constants of the layer
// that uses them.
//
// Scales: one fractional length fl per layer (a dynamic fixed point whose
// exponent is shared by the layer).  With amax the largest alpha, the
// integer length is il = ceil(log2 amax) + 1 and fl = bits - il; a scale is
// A * 2^-fl with A = clamp(rint(alpha * 2^fl), 0, 2^(bits-1) - 1), a signed
// code, so that A * t fits int8.
//
// Layer: with w'[o][k] = A[o][g(k)] * t[o][k] in [-127, 127] the layer is one
// exact int8 product S = sum_k w' q, and y = fp32(double(S) * (double(s_x) *
// 2^-fl)), which is the correctly rounded value of s_x 2^-fl S whenever
// |S| < 2^29.  The planes are written in the folded kernel's fragment order
// with one plane, plus the uint8 offset term 128 * sum_k w' and the
// dequantized scales A * 2^-fl for the direct kernel.
//
// First layer at 8-bit weights (Sec. 4 keeps it at 8w-8a): the weights
// themselves as a signed 8-bit dynamic fixed point with one fractional
// length, fl = 8 - (ceil(log2 max|w|) + 1), W8 = clamp(rint(w * 2^fl),
// -128, 127), in the same prepared layout (W8 as the plane); the layer is
// then computed exactly like the fixed-point-scale layer.
#include <limits.h>

#include "fgq_internal.h"
#include "xlayout.h"

// Every floating-point expression here is evaluated exactly as written.
#pragma clang fp contract(off)

namespace fgq {

PreparedLayout prepared_layout_dfp(int64_t O, int64_t K, int32_t G) {
  PreparedLayout L;
  L.kind = kPrepDfp;
  L.O32 = round_up(O, 32);
  L.Kp = round_up(K, 2 * kFoldKStep);
  L.nks = L.Kp / kFoldKStep;
  L.planes_off = kDfpHeaderBytes;
  L.bias_off = round_up(L.planes_off + L.O32 * L.Kp, 256);
  L.alpha_off = round_up(L.bias_off + 4 * O, 256);
  const int64_t xnb = dfpx_acode_bytes(G);
  const int64_t O128 = round_up(O, 128);
  L.xcodes_off = round_up(L.alpha_off + 4 * O * (K / G), 256);
  L.xacodes_off = round_up(L.xcodes_off + (xnb > 0 ? O128 * L.Kp / 4 : 0), 256);
  L.total = round_up(L.xacodes_off + O128 * (L.Kp / 64) * xnb, 256);
  L.scale_off = L.total;
  return L;
}

namespace {

constexpr int kThreads = 256;
constexpr int kExpThreads = 1024;

// The shared exponent in three launches, accumulated in *fl itself: zero
// it, fold every value into it with an unsigned atomic maximum (a finite
// non-negative float orders as its bit pattern; NaN, Inf or a negative scale
// becomes 0xFFFFFFFF, above every such pattern), then turn the largest value
// into fl (INT32_MIN if any value was rejected).  kSigned: |w| of weights.
__global__ void dfp_exponent_init_kernel(int32_t* __restrict__ fl) { fl[0] = 0; }

template <bool kSigned>
__global__ __launch_bounds__(kExpThreads) void dfp_exponent_kernel(const float* __restrict__ alpha,
                                                                   int64_t n, int32_t* __restrict__ fl) {
  __shared__ uint32_t red[kExpThreads / 64];
  uint32_t vmax = 0;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kExpThreads + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kExpThreads) {
    const float a = kSigned ? fabsf(alpha[i]) : alpha[i];
    const bool ok = a >= 0.0f && a < __builtin_huge_valf();
    const uint32_t v = ok ? __float_as_uint(a + 0.0f) : 0xFFFFFFFFu;  // + 0: -0 becomes +0
    vmax = v > vmax ? v : vmax;
  }
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t o = static_cast<uint32_t>(__shfl_xor(static_cast<int>(vmax), off));
    vmax = o > vmax ? o : vmax;
  }
  if (threadIdx.x % 64 == 0) red[threadIdx.x / 64] = vmax;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 0; i < kExpThreads / 64; ++i) vmax = red[i] > vmax ? red[i] : vmax;
    atomicMax(reinterpret_cast<unsigned int*>(fl), vmax);
  }
}

__global__ void dfp_exponent_final_kernel(int32_t bits, int32_t* __restrict__ fl) {
  const uint32_t v = static_cast<uint32_t>(fl[0]);
  int32_t f = 0;
  const float amax = __uint_as_float(v);
  if (v != 0xFFFFFFFFu && amax > 0.0f) {
    int e;
    const float m = frexpf(amax, &e);  // amax = m 2^e, m in [0.5, 1)
    const int ceil_log2 = m == 0.5f ? e - 1 : e;
    f = bits - (ceil_log2 + 1);
  }
  fl[0] = v == 0xFFFFFFFFu ? INT_MIN : f;
}

template <bool kSigned>
fgq_status launch_exponent(const float* x, int64_t n, int32_t bits, int32_t* fl, hipStream_t st) {
  const int64_t blocks = ceil_div(n, 4 * kExpThreads) < 1024 ? ceil_div(n, 4 * kExpThreads) : 1024;
  hipLaunchKernelGGL(dfp_exponent_init_kernel, dim3(1), dim3(1), 0, st, fl);
  if (n > 0)
    hipLaunchKernelGGL(dfp_exponent_kernel<kSigned>, dim3(static_cast<uint32_t>(blocks)), dim3(kExpThreads), 0, st,
                       x, n, fl);
  hipLaunchKernelGGL(dfp_exponent_final_kernel, dim3(1), dim3(1), 0, st, bits, fl);
  return last_launch();
}

__device__ inline int dfp_code(float alpha, int32_t fl, int32_t bits) {
  const double top = static_cast<double>((1 << (bits - 1)) - 1);
  double v = rint(ldexp(static_cast<double>(alpha), fl));
  v = v > top ? top : v;
  return static_cast<int>(v);
}

__global__ __launch_bounds__(kThreads) void dfp_codes_kernel(const float* __restrict__ alpha, int64_t n,
                                                             int32_t bits, const int32_t* __restrict__ flp,
                                                             int8_t* __restrict__ A) {
  const int32_t fl = *flp;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kThreads)
    A[i] = fl == INT_MIN ? 0 : static_cast<int8_t>(dfp_code(alpha[i], fl, bits));
}

// Byte offset of channel o, reduction index k in the one-plane fragment order.
__device__ inline int64_t frag_offset1(int64_t nks, int64_t o, int64_t k) {
  const int64_t tile = o / 32, ks = k / kFoldKStep;
  const int kk = static_cast<int>(k % kFoldKStep);
  const int half = kk / 32, lane = static_cast<int>(o % 32) + 32 * ((kk % 32) / 16);
  return ((tile * nks + ks) * 2 + half) * 1024 + lane * 16 + (kk % 16);
}

// One block per channel of the padded channel range (O32 for the plane,
// O128 for the expanding GEMM's regions when xnb > 0).
__global__ __launch_bounds__(kThreads) void prepare_dfp_kernel(
    const uint8_t* __restrict__ codes, const float* __restrict__ alpha, int64_t O, int64_t K,
    int32_t G, int32_t bits, int64_t Kp, const int32_t* __restrict__ flp, int8_t* __restrict__ planes,
    int32_t* __restrict__ bias, float* __restrict__ alpha_q, uint8_t* __restrict__ xcodes,
    int8_t* __restrict__ xacodes, int32_t xnb) {
  __shared__ int64_t red[kThreads / 64];
  const int64_t o = blockIdx.x;
  const int64_t nks = Kp / kFoldKStep;
  const int64_t O32 = round_up(O, 32);
  const int32_t fl = *flp;
  const bool live = o < O && fl != INT_MIN;  // else a padding channel (or rejected scales): zeros
  const int64_t ng = K / G;
  const int64_t rb = ceil_div(K, 4);
  auto code = [&](int64_t k) -> uint32_t { return k < K ? (codes[o * rb + k / 4] >> (2 * (k % 4))) & 3u : 0u; };

  // The expanding GEMM's order (xlayout.h): the codes, and the scale codes A.
  if (xnb > 0) {
    const int64_t nk = Kp / 128;
    write_xcodes(codes, o, K, Kp, live, xcodes);
    for (int64_t e = threadIdx.x; e < nk * 2 * xnb; e += kThreads) {
      const int64_t ks = e / (2 * xnb);
      const int hf = static_cast<int>((e / xnb) % 2), j = static_cast<int>(e % xnb);
      const int64_t k = xscale_k(ks, hf, j, G);
      const int A = (live && k < K) ? dfp_code(alpha[o * ng + k / G], fl, bits) : 0;
      xacodes[xfrag_lane(nk, o, ks, hf) * xnb + j] = static_cast<int8_t>(A);
    }
  }
  if (o >= O32) return;
  if (!live) {
    for (int64_t k = threadIdx.x; k < Kp; k += kThreads) planes[frag_offset1(nks, o, k)] = 0;
    return;
  }
  for (int64_t gi = threadIdx.x; gi < ng; gi += kThreads) {
    const int A = dfp_code(alpha[o * ng + gi], fl, bits);
    alpha_q[o * ng + gi] = static_cast<float>(ldexp(static_cast<double>(A), -fl));
  }
  int64_t s = 0;
  for (int64_t k = threadIdx.x; k < Kp; k += kThreads) {
    const uint32_t c = code(k);
    const int t = c == 1 ? 1 : (c == 3 ? -1 : 0);
    const int v = t * (k < K ? dfp_code(alpha[o * ng + k / G], fl, bits) : 0);
    planes[frag_offset1(nks, o, k)] = static_cast<int8_t>(v);
    s += v;
  }
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (threadIdx.x % 64 == 0) red[threadIdx.x / 64] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t v = 0;
    for (int i = 0; i < kThreads / 64; ++i) v += red[i];
    bias[o] = static_cast<int32_t>(128 * v);
  }
}

// First layer at 8-bit weights: one block per channel of the padded range;
// w is [O][C][R][S], k = (r*S + s)*C + c.
__global__ __launch_bounds__(kThreads) void prepare_w8_kernel(
    const float* __restrict__ w, int64_t O, int64_t C, int32_t R, int32_t S, int64_t Kp,
    const int32_t* __restrict__ flp, int8_t* __restrict__ planes, int32_t* __restrict__ bias) {
  __shared__ int64_t red[kThreads / 64];
  const int64_t o = blockIdx.x;
  const int64_t nks = Kp / kFoldKStep;
  const int64_t K = C * R * S;
  const int32_t fl = *flp;
  if (o >= O || fl == INT_MIN) {
    for (int64_t k = threadIdx.x; k < Kp; k += kThreads) planes[frag_offset1(nks, o, k)] = 0;
    return;
  }
  int64_t s = 0;
  for (int64_t k = threadIdx.x; k < Kp; k += kThreads) {
    int v = 0;
    if (k < K) {
      const int64_t c = k % C, rs = k / C;
      const int64_t sx = rs % S, r = rs / S;
      double d = rint(ldexp(static_cast<double>(w[((o * C + c) * R + r) * S + sx]), fl));
      d = d > 127.0 ? 127.0 : (d < -128.0 ? -128.0 : d);
      v = static_cast<int>(d);
    }
    planes[frag_offset1(nks, o, k)] = static_cast<int8_t>(v);
    s += v;
  }
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (threadIdx.x % 64 == 0) red[threadIdx.x / 64] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t v = 0;
    for (int i = 0; i < kThreads / 64; ++i) v += red[i];
    bias[o] = static_cast<int32_t>(128 * v);
  }
}

}  // namespace

fgq_status launch_prepare_w8(const float* w, int64_t O, int64_t C, int32_t R, int32_t S,
                             void* prepared, hipStream_t st) {
  const int64_t K = C * R * S;
  const PreparedLayout L = prepared_layout_dfp(O, K, static_cast<int32_t>(C));
  char* base = static_cast<char*>(prepared);
  int32_t* fl = reinterpret_cast<int32_t*>(base);
  if (launch_exponent<true>(w, O * K, 8, fl, st) != FGQ_OK) return FGQ_ERR_HIP;
  if (L.O32 > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  hipLaunchKernelGGL(prepare_w8_kernel, dim3(static_cast<uint32_t>(L.O32)), dim3(kThreads), 0, st, w, O,
                     C, R, S, L.Kp, fl, reinterpret_cast<int8_t*>(base + L.planes_off),
                     reinterpret_cast<int32_t*>(base + L.bias_off));
  return last_launch();
}

fgq_status launch_dfp_alpha(const float* alpha, int64_t n, int32_t bits, int8_t* A, int32_t* fl,
                            hipStream_t st) {
  if (launch_exponent<false>(alpha, n, bits, fl, st) != FGQ_OK) return FGQ_ERR_HIP;
  if (A && n > 0) {
    const int64_t blocks = ceil_div(n, kThreads) < 4096 ? ceil_div(n, kThreads) : 4096;
    hipLaunchKernelGGL(dfp_codes_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0, st,
                       alpha, n, bits, fl, A);
  }
  return last_launch();
}

fgq_status launch_prepare_dfp(const uint8_t* codes, const float* alpha, int64_t O, int64_t K,
                              int32_t G, int32_t alpha_bits, void* prepared, hipStream_t st) {
  const PreparedLayout L = prepared_layout_dfp(O, K, G);
  char* base = static_cast<char*>(prepared);
  int32_t* fl = reinterpret_cast<int32_t*>(base);
  fgq_status rc = launch_dfp_alpha(alpha, O * (K / G), alpha_bits, nullptr, fl, st);
  if (rc != FGQ_OK) return rc;
  if (L.O32 > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  const int32_t xnb = static_cast<int32_t>(dfpx_acode_bytes(G));
  const int64_t nblk = xnb > 0 ? round_up(O, 128) : L.O32;
  hipLaunchKernelGGL(prepare_dfp_kernel, dim3(static_cast<uint32_t>(nblk)), dim3(kThreads), 0, st,
                     codes, alpha, O, K, G, alpha_bits, L.Kp, fl,
                     reinterpret_cast<int8_t*>(base + L.planes_off),
                     reinterpret_cast<int32_t*>(base + L.bias_off),
                     reinterpret_cast<float*>(base + L.alpha_off),
                     reinterpret_cast<uint8_t*>(base + L.xcodes_off),
                     reinterpret_cast<int8_t*>(base + L.xacodes_off), xnb);
  return last_launch();
}

}  // namespace fgq
