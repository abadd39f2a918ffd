// ternarize.hip -- per-group ternarization (Sec. 3 threshold rule, Eq. (1);
// Sec. 3.1 Eq. (2) and Eq. (5) solved exhaustively; Lemma 1 as method 1)
// and 2-bit packing of the codes.
//
// One 64-lane wave handles a "unit" of U = lcm(G, 4) consecutive reduction
// indices of one output row (several units per wave when U < 64; the last
// unit of a row may be shorter, still a whole number of groups), so every
// code byte is assembled and written by exactly one wave.  Inside a unit:
//   1. each lane loads one weight (w[o][c][r][s] for k = (r*S+s)*C + c),
//   2. ranks inside its group by (decreasing |w|, increasing position),
//   3. one lane per group walks the magnitudes in rank order accumulating
//      S_j in fp64 and f_j = S_j*S_j/j, keeping the first maximum,
//   4. codes t = sign(w) for rank < J are packed four to a byte.
// The fp64 operation sequence matches the plain definition exactly (no
// contraction is possible in it), so alpha/Delta/codes are reproducible
// bit for bit on any IEEE machine.
#include "fgq_internal.h"

// Every floating-point expression here is evaluated exactly as written.
#pragma clang fp contract(off)

namespace fgq {
namespace {

constexpr int kWave = 64;

__device__ inline int code_of(float w, bool keep) {
  if (!keep) return 0;
  return w > 0.0f ? 1 : (w < 0.0f ? 3 : 0);
}

__global__ __launch_bounds__(kWave) void ternarize_kernel(
    const float* __restrict__ w, int64_t C, int32_t R, int32_t S, int32_t G,
    int64_t K, int32_t U, int32_t upw, int64_t nunits, int32_t method,
    uint8_t* __restrict__ codes, float* __restrict__ alpha,
    float* __restrict__ delta) {
  extern __shared__ unsigned char smem[];
  const int NE = upw * U;  // elements handled by this wave
  float* mag = reinterpret_cast<float*>(smem);         // [NE] |w| in position order
  float* sorted = mag + NE;                             // [NE] |w| in rank order per group
  float* sgn = sorted + NE;                             // [NE] w (for its sign)
  int* rank = reinterpret_cast<int*>(sgn + NE);         // [NE]
  int* bad = rank + NE;                                 // [NE] non-finite flag
  float* gthr = reinterpret_cast<float*>(bad + NE);     // [NE/G] Lemma threshold
  int* gJ = reinterpret_cast<int*>(gthr + NE / G);      // [NE/G] kept count
  unsigned char* cbyte = reinterpret_cast<unsigned char*>(gJ + NE / G);  // [NE]

  const int lane = threadIdx.x;
  const int64_t unit0 = static_cast<int64_t>(blockIdx.x) * upw;
  const int64_t units_per_row = ceil_div(K, U);

  // 1. load
  for (int e = lane; e < NE; e += kWave) {
    const int64_t u = unit0 + e / U;
    float v = 0.0f;
    int isbad = 0;
    const int64_t k = (u % units_per_row) * U + e % U;
    if (u < nunits && k < K) {
      const int64_t o = u / units_per_row;
      const int64_t c = k % C;
      const int64_t rs = k / C;
      const int64_t s = rs % S;
      const int64_t r = rs / S;
      v = w[((o * C + c) * R + r) * S + s];
      isbad = isfinite(v) ? 0 : 1;
    }
    mag[e] = fabsf(v);
    sgn[e] = v;
    bad[e] = isbad;
  }
  __syncthreads();

  // 2. rank inside the group (decreasing magnitude, then increasing position)
  for (int e = lane; e < NE; e += kWave) {
    const int gb = (e / G) * G;
    const float a = mag[e];
    int rk = 0;
    for (int j = gb; j < gb + G; ++j) {
      const float b = mag[j];
      rk += (b > a || (b == a && j < e)) ? 1 : 0;
    }
    rank[e] = rk;
    sorted[gb + rk] = a;
  }
  __syncthreads();

  // 3. one lane per group: the exhaustive search of Eq. (5) (or Lemma 1)
  const int ngw = NE / G;
  for (int gi = lane; gi < ngw; gi += kWave) {
    const int gb = gi * G;
    const int64_t u = unit0 + gb / U;
    const int64_t k0 = (u % units_per_row) * U + (gb % U);
    if (u >= nunits || k0 >= K) {
      gJ[gi] = 0;
      gthr[gi] = 0.0f;
      continue;
    }
    int anybad = 0;
    for (int j = gb; j < gb + G; ++j) anybad |= bad[j];
    const int64_t o = u / units_per_row;
    const int64_t gidx = o * (K / G) + k0 / G;
    float a_out, d_out;
    int J = 0;
    float thr = 0.0f;
    if (anybad) {
      a_out = __builtin_nanf("");
      d_out = __builtin_nanf("");
    } else if (method == FGQ_TERN_EXACT) {
      double Ssum = 0.0, bestS = 0.0, bestf = 0.0;
      for (int j = 1; j <= G; ++j) {
        const float a = sorted[gb + j - 1];
        if (!(a > 0.0f)) break;
        Ssum = Ssum + static_cast<double>(a);
        const double f = (Ssum * Ssum) / static_cast<double>(j);
        if (f > bestf) {
          bestf = f;
          bestS = Ssum;
          J = j;
        }
      }
      a_out = J > 0 ? static_cast<float>(bestS / static_cast<double>(J)) : 0.0f;
      d_out = J < G ? sorted[gb + J] : 0.0f;
    } else {  // Lemma 1: Delta = mean |w|
      double Ssum = 0.0;
      for (int j = gb; j < gb + G; ++j) Ssum = Ssum + static_cast<double>(mag[j]);
      thr = static_cast<float>(Ssum / static_cast<double>(G));
      double Ksum = 0.0;
      int cnt = 0;
      for (int j = gb; j < gb + G; ++j) {
        if (mag[j] > thr) {
          Ksum = Ksum + static_cast<double>(mag[j]);
          ++cnt;
        }
      }
      a_out = cnt > 0 ? static_cast<float>(Ksum / static_cast<double>(cnt)) : 0.0f;
      d_out = thr;
    }
    alpha[gidx] = a_out;
    if (delta) delta[gidx] = d_out;
    gJ[gi] = anybad ? 0 : J;
    gthr[gi] = anybad ? __builtin_inff() : thr;
  }
  __syncthreads();

  // 4. codes, four to a byte
  for (int e = lane; e < NE; e += kWave) {
    const int gi = e / G;
    const bool keep = (method == FGQ_TERN_EXACT) ? (rank[e] < gJ[gi]) : (mag[e] > gthr[gi]);
    cbyte[e] = static_cast<unsigned char>(code_of(sgn[e], keep));
  }
  __syncthreads();
  const int64_t rb = ceil_div(K, 4);
  for (int b = lane; b < NE / 4; b += kWave) {
    const int64_t u = unit0 + (4 * b) / U;
    const int64_t k = (u % units_per_row) * U + (4 * b) % U;
    if (u >= nunits || k >= K) continue;
    const int64_t o = u / units_per_row;
    const unsigned v = cbyte[4 * b] | (cbyte[4 * b + 1] << 2) | (cbyte[4 * b + 2] << 4) |
                       (cbyte[4 * b + 3] << 6);
    codes[o * rb + k / 4] = static_cast<uint8_t>(v);
  }
}

int gcd_i(int a, int b) {
  while (b) {
    int t = a % b;
    a = b;
    b = t;
  }
  return a;
}

}  // namespace

fgq_status launch_ternarize(const float* w, int64_t O, int64_t C, int32_t R,
                            int32_t S, int32_t G, int32_t method,
                            uint8_t* codes, float* alpha, float* delta,
                            hipStream_t st) {
  const int64_t K = static_cast<int64_t>(R) * S * C;
  const int32_t U = G / gcd_i(G, 4) * 4;  // lcm(G, 4)
  const int32_t upw = U >= kWave ? 1 : kWave / U;
  const int32_t NE = upw * U;
  const int64_t nunits = O * ceil_div(K, U);
  const size_t smem = static_cast<size_t>(NE) * (4 * 3 + 4 * 2 + 1) +
                      static_cast<size_t>(NE / G) * 8 + 16;
  if (smem > 64 * 1024) return FGQ_ERR_UNSUPPORTED;
  const int64_t grid = ceil_div(nunits, upw);
  if (grid > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  hipLaunchKernelGGL(ternarize_kernel, dim3(static_cast<uint32_t>(grid)), dim3(kWave), smem, st,
                     w, C, R, S, G, K, U, upw, nunits, method, codes, alpha, delta);
  return last_launch();
}

}  // namespace fgq
