// ternarize.hip -- per-group ternarization (Sec. 3 threshold rule, Eq. (1);
// Sec. 3.1 Eq. (2) and Eq. (5) solved exhaustively; Lemma 1 as method 1;
// the Gaussian-optimal threshold as method 3; Eq. (3)-(4), asymmetric
// thresholds solved exhaustively; the K-S distances that choose between the
// Gaussian and exponential references per layer) and 2-bit packing.
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

// Root of 2u (1 - Phi(u)) = phi(u): for w ~ N(0, sigma) the expected Eq. (5)
// objective of the threshold u*sigma is proportional to
// phi(u)^2 / (1 - Phi(u)), which peaks there.
constexpr double kGaussU = 0.61200318096248076;

__device__ inline int code_of(float w, bool keep) {
  if (!keep) return 0;
  return w > 0.0f ? 1 : (w < 0.0f ? 3 : 0);
}

__global__ __launch_bounds__(kWave) void ternarize_kernel(
    const float* __restrict__ w, int64_t C, int32_t R, int32_t S, int32_t G,
    int64_t K, int32_t U, int32_t upw, int64_t nunits, int32_t method,
    uint8_t* __restrict__ codes, float* __restrict__ alpha,
    float* __restrict__ delta, float* __restrict__ delta_n) {
  extern __shared__ unsigned char smem[];
  const int NE = upw * U;  // elements handled by this wave
  const bool asym = method == kTernAsym;
  const int NA = asym ? NE : 0;  // the asymmetric search's arrays
  float* mag = reinterpret_cast<float*>(smem);         // [NE] |w| in position order
  float* sorted = mag + NE;                             // [NE] |w| in rank order per group
  float* sgn = sorted + NE;                             // [NE] w (for its sign)
  float* spos = sgn + NE;                               // [NA] positive |w|, rank order per group
  float* sneg = spos + NA;                              // [NA] negative |w|, rank order per group
  int* rank = reinterpret_cast<int*>(sneg + NA);        // [NE]
  int* srank = rank + NE;                               // [NA] rank among same-sign weights
  int* bad = srank + NA;                                // [NE] non-finite flag
  float* gthr = reinterpret_cast<float*>(bad + NE);     // [NE/G] threshold rules
  int* gJ = reinterpret_cast<int*>(gthr + NE / G);      // [NE/G] kept count (exact; asym positives)
  int* gJn = gJ + NE / G;                               // [NE/G] asym: kept negatives
  unsigned char* cbyte = reinterpret_cast<unsigned char*>(gJn + NE / G);  // [NE]

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

  // 2. rank inside the group (decreasing magnitude, then increasing
  // position), overall and among the weights of the same sign
  for (int e = lane; e < NE; e += kWave) {
    const int gb = (e / G) * G;
    const float a = mag[e];
    const int se = sgn[e] > 0.0f ? 1 : (sgn[e] < 0.0f ? -1 : 0);
    int rk = 0, srk = 0;
    for (int j = gb; j < gb + G; ++j) {
      const float b = mag[j];
      const int before = (b > a || (b == a && j < e)) ? 1 : 0;
      const int sj = sgn[j] > 0.0f ? 1 : (sgn[j] < 0.0f ? -1 : 0);
      rk += before;
      srk += (sj == se) ? before : 0;
    }
    rank[e] = rk;
    sorted[gb + rk] = a;
    if (asym) {
      srank[e] = srk;
      if (se > 0) spos[gb + srk] = a;
      if (se < 0) sneg[gb + srk] = a;
    }
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
      gJn[gi] = 0;
      gthr[gi] = 0.0f;
      continue;
    }
    int anybad = 0;
    for (int j = gb; j < gb + G; ++j) anybad |= bad[j];
    const int64_t o = u / units_per_row;
    const int64_t gidx = o * (K / G) + k0 / G;
    float a_out, d_out, dn_out = 0.0f;
    int J = 0, Jn = 0;
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
    } else if (method == kTernAsym) {
      // Eq. (3)-(4): every pair (a, b) of prefixes of the positive and the
      // negative magnitudes in rank order; P_a and N_b are fp64 prefix sums,
      // f = (P_a + N_b)^2 / (a + b), the first maximum (a, then b) is kept
      int np = 0, nn = 0;
      for (int j = gb; j < gb + G; ++j) {
        np += sgn[j] > 0.0f ? 1 : 0;
        nn += sgn[j] < 0.0f ? 1 : 0;
      }
      double Pa = 0.0, bestf = 0.0, bestT = 0.0;
      for (int a = 0; a <= np; ++a) {
        if (a > 0) Pa = Pa + static_cast<double>(spos[gb + a - 1]);
        double Nb = 0.0;
        for (int b = 0; b <= nn; ++b) {
          if (b > 0) Nb = Nb + static_cast<double>(sneg[gb + b - 1]);
          if (a + b == 0) continue;
          const double T = Pa + Nb;
          const double f = (T * T) / static_cast<double>(a + b);
          if (f > bestf) {
            bestf = f;
            bestT = T;
            J = a;
            Jn = b;
          }
        }
      }
      a_out = J + Jn > 0 ? static_cast<float>(bestT / static_cast<double>(J + Jn)) : 0.0f;
      d_out = J < np ? spos[gb + J] : 0.0f;
      dn_out = Jn < nn ? sneg[gb + Jn] : 0.0f;
    } else {
      if (method == FGQ_TERN_GAUSS) {  // Delta = kGaussU * rms(w)
        double Q = 0.0;
        for (int j = gb; j < gb + G; ++j) {
          const double v = static_cast<double>(sgn[j]);
          Q = Q + v * v;
        }
        thr = static_cast<float>(kGaussU * sqrt(Q / static_cast<double>(G)));
      } else {  // Lemma 1: Delta = mean |w|
        double Ssum = 0.0;
        for (int j = gb; j < gb + G; ++j) Ssum = Ssum + static_cast<double>(mag[j]);
        thr = static_cast<float>(Ssum / static_cast<double>(G));
      }
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
    if (delta_n) delta_n[gidx] = anybad ? __builtin_nanf("") : dn_out;
    gJ[gi] = anybad ? 0 : J;
    gJn[gi] = anybad ? 0 : Jn;
    gthr[gi] = anybad ? __builtin_inff() : thr;
  }
  __syncthreads();

  // 4. codes, four to a byte
  for (int e = lane; e < NE; e += kWave) {
    const int gi = e / G;
    bool keep;
    if (method == FGQ_TERN_EXACT)
      keep = rank[e] < gJ[gi];
    else if (method == kTernAsym)
      keep = (sgn[e] > 0.0f && srank[e] < gJ[gi]) || (sgn[e] < 0.0f && srank[e] < gJn[gi]);
    else
      keep = mag[e] > gthr[gi];
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

// Sec. 3.1: K-S distances of the weight magnitudes to the half-normal law of
// N(0, sigma) (sigma = rms) and to the exponential law of scale mu = mean|w|
// (1/lambda of Lemma 1), both fitted by maximum likelihood, on at most
// kKsSample magnitudes (every s-th weight in storage order,
// s = ceil(n / kKsSample)).  One workgroup: the sample is sorted ascending in
// LDS (bitonic), sigma^2 and mu are fp64 sums in ascending order by one
// thread, and D = max_i max(i/ns - F(m_(i)), F(m_(i)) - (i-1)/ns) is a
// maximum over threads (exact in any order).  A sample of zeros gives D = 0.
// d (nullable): [D_gauss, D_exp]; pick (nullable): the threshold rule the
// layer takes, FGQ_TERN_EXP_LEMMA when the exponential law is strictly
// closer, else FGQ_TERN_GAUSS.
constexpr int kKsThreads = 1024;

__global__ __launch_bounds__(kKsThreads) void ks_kernel(const float* __restrict__ w, int64_t n,
                                                        double* __restrict__ d, int32_t* __restrict__ pick) {
  __shared__ float m[kKsSample];
  __shared__ double part[2][kKsThreads / 64];
  __shared__ double mom[2];
  const int tid = threadIdx.x;
  const int64_t step = (n + kKsSample - 1) / kKsSample;
  const int ns = static_cast<int>((n + step - 1) / step);
  int P = 1;
  while (P < ns) P <<= 1;
  for (int i = tid; i < P; i += kKsThreads) m[i] = i < ns ? fabsf(w[i * step]) : __builtin_inff();
  __syncthreads();
  for (int k = 2; k <= P; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < P; i += kKsThreads) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const float a = m[i], b = m[ixj];
          if ((a > b) == ((i & k) == 0)) {
            m[i] = b;
            m[ixj] = a;
          }
        }
      }
      __syncthreads();
    }
  if (tid == 0) {
    double Q = 0.0, S = 0.0;
    for (int i = 0; i < ns; ++i) {
      const double v = static_cast<double>(m[i]);
      Q = Q + v * v;
      S = S + v;
    }
    mom[0] = sqrt(Q / static_cast<double>(ns));
    mom[1] = S / static_cast<double>(ns);
  }
  __syncthreads();
  const double sigma = mom[0], mu = mom[1];
  double dg = 0.0, de = 0.0;
  if (mu > 0.0) {
    for (int i = tid; i < ns; i += kKsThreads) {
      const double x = static_cast<double>(m[i]);
      const double hi = static_cast<double>(i + 1) / static_cast<double>(ns);
      const double lo = static_cast<double>(i) / static_cast<double>(ns);
      const double fg = erf(x / (sigma * sqrt(2.0)));
      const double fe = 1.0 - exp(-x / mu);
      dg = fmax(dg, fmax(hi - fg, fg - lo));
      de = fmax(de, fmax(hi - fe, fe - lo));
    }
  }
  for (int off = 32; off > 0; off >>= 1) {
    dg = fmax(dg, __shfl_xor(dg, off));
    de = fmax(de, __shfl_xor(de, off));
  }
  if (tid % 64 == 0) {
    part[0][tid / 64] = dg;
    part[1][tid / 64] = de;
  }
  __syncthreads();
  if (tid == 0) {
    for (int i = 0; i < kKsThreads / 64; ++i) {
      dg = fmax(dg, part[0][i]);
      de = fmax(de, part[1][i]);
    }
    if (d) {
      d[0] = dg;
      d[1] = de;
    }
    if (pick) pick[0] = de < dg ? FGQ_TERN_EXP_LEMMA : FGQ_TERN_GAUSS;
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

fgq_status launch_ks(const float* w, int64_t n, double* d, int32_t* pick, hipStream_t st) {
  hipLaunchKernelGGL(ks_kernel, dim3(1), dim3(kKsThreads), 0, st, w, n, d, pick);
  return last_launch();
}

fgq_status launch_ternarize(const float* w, int64_t O, int64_t C, int32_t R,
                            int32_t S, int32_t G, int32_t method,
                            uint8_t* codes, float* alpha, float* delta, float* delta_n,
                            hipStream_t st) {
  const int64_t K = static_cast<int64_t>(R) * S * C;
  const int32_t U = G / gcd_i(G, 4) * 4;  // lcm(G, 4)
  const int32_t upw = U >= kWave ? 1 : kWave / U;
  const int32_t NE = upw * U;
  const int64_t nunits = O * ceil_div(K, U);
  const size_t NA = method == kTernAsym ? NE : 0;
  const size_t smem = static_cast<size_t>(NE) * (4 * 3 + 4 * 2 + 1) + NA * 12 +
                      static_cast<size_t>(NE / G) * 12 + 16;
  if (smem > 64 * 1024) return FGQ_ERR_UNSUPPORTED;
  const int64_t grid = ceil_div(nunits, upw);
  if (grid > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  hipLaunchKernelGGL(ternarize_kernel, dim3(static_cast<uint32_t>(grid)), dim3(kWave), smem, st,
                     w, C, R, S, G, K, U, upw, nunits, method, codes, alpha, delta, delta_n);
  return last_launch();
}

}  // namespace fgq
