// exact.hip -- direct per-group FGQ layer kernels.
//
// exact_conv: y = s_x * sum_g alpha_g * P_g with every group sum P_g formed
//   exactly in int32 (v_dot4 on four codes and four activations at a time)
//   and the alpha-weighted sum accumulated in fp64 in group order, then
//   rounded once to fp32.  Every fp64 product alpha*P is exact (24 + 15
//   bits), so the result equals the plain definition's fp64 evaluation bit
//   for bit.  This is the general path (any G, C, stride, padding, bits)
//   and the "v_dot4 VALU" variant of the G=4 layer.
// group_sums: the int32 P_g themselves for a range of output rows.
//
// uint8 activations are signed-offset (q ^ 0x80 = q - 128) so that the
// signed v_dot4_i32_i8 applies; P_g = P'_g + 128*T_g with T_g the sum of the
// group's codes, accumulated alongside.  Out-of-image taps read q = 0, i.e.
// q' = -128, so the identity also holds there.
#include "fgq_internal.h"
#include "qcode.h"

// Every floating-point expression here is evaluated exactly as written.
#pragma clang fp contract(off)

namespace fgq {
namespace {

constexpr int kTM = 64, kTO = 64, kKC = 64;
constexpr int kStride = kKC + 4;  // LDS row stride in bytes (bank spread)

__device__ inline uint32_t unpack_code_byte(uint32_t b) {
  // 4 two-bit codes -> 4 int8 in {-1,0,1}: spread to bytes, sign-extend.
  uint32_t x = (b & 3u) | ((b & 0xCu) << 6) | ((b & 0x30u) << 12) | ((b & 0xC0u) << 18);
  uint32_t hi = x & 0x02020202u;
  return x | (hi * 0x7Eu);
}

__device__ inline unsigned act_elem(const uint8_t* __restrict__ q, int bits, int64_t e) {
  if (bits == 8) return q[e];
  return (q[e >> 1] >> (4 * (e & 1))) & 15u;
}

// Element index of A[m][k] in the NHWC activation tensor, or -1 outside.
__device__ inline int64_t a_index(const ConvGeom& g, int64_t m, int64_t k) {
  const int64_t wo = m % g.Wo;
  const int64_t t = m / g.Wo;
  const int64_t ho = t % g.Ho;
  const int64_t b = t / g.Ho;
  const int64_t c = k % g.C;
  const int64_t rs = k / g.C;
  const int64_t s = rs % g.S;
  const int64_t r = rs / g.S;
  const int64_t hi = ho * g.sh - g.ph + r;
  const int64_t wi = wo * g.sw - g.pw + s;
  if (hi < 0 || hi >= g.H || wi < 0 || wi >= g.W) return -1;
  return ((b * g.H + hi) * g.W + wi) * g.C + c;
}

// kVec: C % 4 == 0, so four consecutive k share one tap and are contiguous.
template <int kBits, bool kVec, bool kDot4, int kOut>
__global__ __launch_bounds__(256) void exact_conv_kernel(
    const uint8_t* __restrict__ q, const float* __restrict__ sxp,
    const uint8_t* __restrict__ codes, const float* __restrict__ alpha,
    ConvGeom g, LayerOut out) {
  __shared__ __attribute__((aligned(16))) int8_t As[kTM * kStride];
  __shared__ __attribute__((aligned(16))) int8_t Ts[kTO * kStride];
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int64_t m0 = static_cast<int64_t>(blockIdx.x) * kTM;
  const int64_t o0 = static_cast<int64_t>(blockIdx.y) * kTO;
  const int64_t ng = g.K / g.G;
  const int64_t rb = ceil_div(g.K, 4);
  const uint32_t xor_mask = kBits == 8 ? 0x80808080u : 0u;

  double acc[4][4];
  int32_t P[4][4];
  int32_t T[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    T[i] = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      acc[i][j] = 0.0;
      P[i][j] = 0;
    }
  }

  for (int64_t kc = 0; kc < g.K; kc += kKC) {
    // ---- activation tile A[64][64] (int8, offset for u8) ----
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int wid = tid + 256 * it;      // 1024 words of 4 k
      const int r = wid / 16, wd = wid % 16;
      const int64_t m = m0 + r;
      const int64_t k = kc + 4 * wd;
      uint32_t word = 0;
      if (m < g.M) {
        if (kVec) {
          if (k < g.K) {
            const int64_t e = a_index(g, m, k);
            if (e >= 0) {
              if (kBits == 8) {
                word = *reinterpret_cast<const uint32_t*>(q + e);
              } else {
                const uint32_t h = *reinterpret_cast<const uint16_t*>(q + e / 2);
                word = (h & 0xFu) | ((h & 0xF0u) << 4) | ((h & 0xF00u) << 8) | ((h & 0xF000u) << 12);
              }
            }
          }
        } else {
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            if (k + b < g.K) {
              const int64_t e = a_index(g, m, k + b);
              if (e >= 0) word |= act_elem(q, kBits, e) << (8 * b);
            }
          }
        }
      }
      *reinterpret_cast<uint32_t*>(&As[r * kStride + 4 * wd]) = word ^ xor_mask;
    }
    // ---- code tile T[64][64] (int8 in {-1,0,1}) ----
    {
      const int col = tid / 4, part = tid % 4;  // 4 code bytes per thread
      const int64_t o = o0 + col;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int64_t byte = kc / 4 + part * 4 + b;
        uint32_t cb = 0;
        if (o < g.O && byte < rb) cb = codes[o * rb + byte];
        *reinterpret_cast<uint32_t*>(&Ts[col * kStride + 4 * (part * 4 + b)]) = unpack_code_byte(cb);
      }
    }
    __syncthreads();

    const int64_t kend = (g.K - kc) < kKC ? (g.K - kc) : kKC;
    if (kDot4) {
      // G % 4 == 0: groups end on word boundaries.
      for (int wd = 0; wd < kKC / 4; ++wd) {
        if (4 * wd >= kend) break;
        int32_t a[4], t[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const int32_t*>(&As[(ty + 16 * i) * kStride + 4 * wd]);
#pragma unroll
        for (int j = 0; j < 4; ++j) t[j] = *reinterpret_cast<const int32_t*>(&Ts[(tx + 16 * j) * kStride + 4 * wd]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) P[i][j] = __builtin_amdgcn_sdot4(a[i], t[j], P[i][j], false);
        if (kBits == 8) {
#pragma unroll
          for (int j = 0; j < 4; ++j) T[j] = __builtin_amdgcn_sdot4(t[j], 0x01010101, T[j], false);
        }
        const int64_t kn = kc + 4 * wd + 4;
        if (kn % g.G == 0) {
          const int64_t gi = kn / g.G - 1;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int64_t o = o0 + tx + 16 * j;
            const double al = o < g.O ? static_cast<double>(alpha[o * ng + gi]) : 0.0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int32_t pt = P[i][j] + 128 * T[j];
              acc[i][j] = fma(al, static_cast<double>(pt), acc[i][j]);
              P[i][j] = 0;
            }
            T[j] = 0;
          }
        }
      }
    } else {
      for (int kk = 0; kk < kKC; ++kk) {
        if (kk >= kend) break;
        int32_t a[4], t[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = As[(ty + 16 * i) * kStride + kk];
#pragma unroll
        for (int j = 0; j < 4; ++j) t[j] = Ts[(tx + 16 * j) * kStride + kk];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) P[i][j] += a[i] * t[j];
        if (kBits == 8) {
#pragma unroll
          for (int j = 0; j < 4; ++j) T[j] += t[j];
        }
        const int64_t kn = kc + kk + 1;
        if (kn % g.G == 0) {
          const int64_t gi = kn / g.G - 1;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int64_t o = o0 + tx + 16 * j;
            const double al = o < g.O ? static_cast<double>(alpha[o * ng + gi]) : 0.0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int32_t pt = P[i][j] + 128 * T[j];
              acc[i][j] = fma(al, static_cast<double>(pt), acc[i][j]);
              P[i][j] = 0;
            }
            T[j] = 0;
          }
        }
      }
    }
    __syncthreads();
  }

  const double sx = static_cast<double>(*sxp);
  with_out_scale<kOut>(out.scale, [&](const QScale& qs, auto rcp) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t m = m0 + ty + 16 * i;
      if (m >= g.M) continue;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t o = o0 + tx + 16 * j;  // lanes tx and tx^1 hold channels o and o^1
        if (o < g.O)
          emit_out<kOut, decltype(rcp)::value>(out.y, out.q, qs, m * g.O + o, g.M * g.O, static_cast<int>(o),
                                               static_cast<float>(sx * acc[i][j]), out.res);
      }
    }
  });
}

// One thread per (row, o, g): P = sum over the group of t * q, exact.
template <int kBits>
__global__ __launch_bounds__(256) void group_sums_kernel(
    const uint8_t* __restrict__ q, const uint8_t* __restrict__ codes, ConvGeom g,
    int64_t row0, int64_t nrows, int32_t* __restrict__ P) {
  const int64_t ng = g.K / g.G;
  const int64_t total = nrows * g.O * ng;
  const int64_t rb = ceil_div(g.K, 4);
  for (int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; idx < total;
       idx += static_cast<int64_t>(gridDim.x) * 256) {
    const int64_t gi = idx % ng;
    const int64_t o = (idx / ng) % g.O;
    const int64_t m = row0 + idx / (ng * g.O);
    int32_t acc = 0;
    for (int64_t k = gi * g.G; k < (gi + 1) * g.G; ++k) {
      const uint32_t c = (codes[o * rb + k / 4] >> (2 * (k % 4))) & 3u;
      if (c == 0) continue;
      const int64_t e = a_index(g, m, k);
      const int32_t a = e >= 0 ? static_cast<int32_t>(act_elem(q, kBits, e)) : 0;
      acc += c == 1 ? a : -a;
    }
    P[idx] = acc;
  }
}

template <int kBits, int kOut>
fgq_status launch_exact_out(const uint8_t* q, const float* sx, const uint8_t* codes,
                            const float* alpha, const ConvGeom& g, const LayerOut& y, hipStream_t st) {
  const int64_t gx = ceil_div(g.M, kTM), gy = ceil_div(g.O, kTO);
  if (gx > 0x7fffffffLL || gy > 65535) return FGQ_ERR_SHAPE;
  const dim3 grid(static_cast<uint32_t>(gx), static_cast<uint32_t>(gy));
  const bool vec = (g.C % 4 == 0) && (reinterpret_cast<uintptr_t>(q) % 4 == 0);
  const bool dot4 = g.G % 4 == 0;
  if (vec && dot4)
    hipLaunchKernelGGL((exact_conv_kernel<kBits, true, true, kOut>), grid, dim3(256), 0, st, q, sx, codes, alpha, g, y);
  else if (dot4)
    hipLaunchKernelGGL((exact_conv_kernel<kBits, false, true, kOut>), grid, dim3(256), 0, st, q, sx, codes, alpha, g, y);
  else if (vec)
    hipLaunchKernelGGL((exact_conv_kernel<kBits, true, false, kOut>), grid, dim3(256), 0, st, q, sx, codes, alpha, g, y);
  else
    hipLaunchKernelGGL((exact_conv_kernel<kBits, false, false, kOut>), grid, dim3(256), 0, st, q, sx, codes, alpha, g, y);
  return last_launch();
}

template <int kBits>
fgq_status launch_exact_bits(const uint8_t* q, const float* sx, const uint8_t* codes,
                             const float* alpha, const ConvGeom& g, const LayerOut& y, hipStream_t st) {
  switch (y.bits) {
    case 0: return launch_exact_out<kBits, 0>(q, sx, codes, alpha, g, y, st);
    case 2: return launch_exact_out<kBits, 2>(q, sx, codes, alpha, g, y, st);
    case 2 | 8: return launch_exact_out<kBits, 2 | 8>(q, sx, codes, alpha, g, y, st);
    case 2 | 4: return launch_exact_out<kBits, 2 | 4>(q, sx, codes, alpha, g, y, st);
    case 8: return launch_exact_out<kBits, 8>(q, sx, codes, alpha, g, y, st);
    default: return launch_exact_out<kBits, 4>(q, sx, codes, alpha, g, y, st);
  }
}

}  // namespace

fgq_status launch_exact_conv(const uint8_t* q, const float* sx, const uint8_t* codes,
                             const float* alpha, const ConvGeom& g, const LayerOut& y, hipStream_t st) {
  return g.bits == 8 ? launch_exact_bits<8>(q, sx, codes, alpha, g, y, st)
                     : launch_exact_bits<4>(q, sx, codes, alpha, g, y, st);
}

fgq_status launch_group_sums(const uint8_t* q, const uint8_t* codes, const ConvGeom& g,
                             int64_t row0, int64_t nrows, int32_t* P, hipStream_t st) {
  const int64_t total = nrows * g.O * (g.K / g.G);
  if (total == 0) return FGQ_OK;
  int64_t blocks = ceil_div(total, 256);
  if (blocks > 65536) blocks = 65536;
  if (g.bits == 8)
    hipLaunchKernelGGL(group_sums_kernel<8>, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0, st, q, codes, g, row0, nrows, P);
  else
    hipLaunchKernelGGL(group_sums_kernel<4>, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0, st, q, codes, g, row0, nrows, P);
  return last_launch();
}

}  // namespace fgq
