/*
 * fgq_oracle.c -- plain, slow, obviously-correct CPU oracle for FGQ
 * inference.  TEST INFRASTRUCTURE ONLY: no product code includes, links or
 * calls it.  Build: gcc -O2 -fno-fast-math -ffp-contract=off -fopenmp.
 * See fgq_oracle.h for the conventions and the passages each part follows.
 */
#include "fgq_oracle.h"

#include <math.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Ternarization (Sec. 3, Eq. (1); Sec. 3.1, Eq. (2), Eq. (5))               */
/* ------------------------------------------------------------------------ */

typedef struct {
  float a;      /* |w_i| */
  int64_t idx;  /* position inside the group */
} mag_t;

/* Order by decreasing magnitude, ties by increasing index. */
static int cmp_mag(const void* pa, const void* pb) {
  const mag_t* x = (const mag_t*)pa;
  const mag_t* y = (const mag_t*)pb;
  if (x->a > y->a) return -1;
  if (x->a < y->a) return 1;
  if (x->idx < y->idx) return -1;
  if (x->idx > y->idx) return 1;
  return 0;
}

static float sign_of(float v) { return v > 0.0f ? 1.0f : (v < 0.0f ? -1.0f : 0.0f); }

/*
 * Eq. (5): for a candidate threshold the kept set I_Delta is {i : |w_i| >
 * Delta}; alpha = sum_{I_Delta}|w| / |I_Delta| and Delta* maximises
 * (sum_{I_Delta}|w|)^2 / |I_Delta|.  Every distinct kept set is a prefix of
 * the magnitudes sorted in decreasing order, so the exhaustive ("brute
 * force", Sec. 3.1) search visits the prefixes j = 1..n of non-zero
 * magnitudes: S_j = S_{j-1} + a_(j) (fp64, in sorted order) and
 * f_j = S_j * S_j / j.  J is the first j reaching the maximum (strict >).
 * alpha = fp32(S_J / J) at the best prefix length J; Delta = a_(J+1), the
 * largest pruned magnitude (0 when nothing is pruned); codes t_i = sign(w_i)
 * for the J largest magnitudes.
 */
static int ternarize_exact(const float* w, int64_t n, int64_t stride, int8_t* t,
                           int64_t tstride, float* alpha, float* delta) {
  mag_t* m = (mag_t*)malloc(sizeof(mag_t) * (size_t)(n > 0 ? n : 1));
  if (!m) return ORC_ERR_SHAPE;
  for (int64_t i = 0; i < n; ++i) {
    m[i].a = fabsf(w[i * stride]);
    m[i].idx = i;
  }
  qsort(m, (size_t)n, sizeof(mag_t), cmp_mag);

  double S = 0.0, bestS = 0.0, bestf = 0.0;
  int64_t jstar = 0;
  for (int64_t j = 1; j <= n; ++j) {
    float a = m[j - 1].a;
    if (!(a > 0.0f)) break; /* zeros are never kept (Sec. 3.1) */
    S = S + (double)a;
    double f = (S * S) / (double)j;
    if (f > bestf) {
      bestf = f;
      bestS = S;
      jstar = j;
    }
  }
  *alpha = jstar > 0 ? (float)(bestS / (double)jstar) : 0.0f;
  *delta = jstar < n ? m[jstar].a : 0.0f;
  for (int64_t i = 0; i < n; ++i) t[i * tstride] = 0;
  for (int64_t j = 0; j < jstar; ++j) {
    int64_t i = m[j].idx;
    t[i * tstride] = (int8_t)sign_of(w[i * stride]);
  }
  free(m);
  return ORC_OK;
}

/*
 * Lemma 1: if |W| follows an exponential law, Delta* is approximately
 * 1/lambda, the mean magnitude.  Delta = fp32(sum|w| / n) (fp64 sum in index
 * order), kept set {i : |w_i| > Delta} compared in fp32, alpha = fp32(mean
 * of the kept magnitudes) as in Eq. (5).
 */
static int ternarize_lemma(const float* w, int64_t n, int64_t stride, int8_t* t,
                           int64_t tstride, float* alpha, float* delta) {
  double S = 0.0;
  for (int64_t i = 0; i < n; ++i) S = S + (double)fabsf(w[i * stride]);
  float d = (float)(S / (double)n);
  double K = 0.0;
  int64_t cnt = 0;
  for (int64_t i = 0; i < n; ++i) {
    float a = fabsf(w[i * stride]);
    if (a > d) {
      K = K + (double)a;
      cnt += 1;
      t[i * tstride] = (int8_t)sign_of(w[i * stride]);
    } else {
      t[i * tstride] = 0;
    }
  }
  *alpha = cnt > 0 ? (float)(K / (double)cnt) : 0.0f;
  *delta = d;
  return ORC_OK;
}

/*
 * Gaussian reference (Sec. 3.1, the distribution the K-S test may select):
 * for w ~ N(0, sigma) and a threshold u*sigma, the expected objective of
 * Eq. (5), E[|w|; |w| > u sigma]^2 / P(|w| > u sigma), is proportional to
 * phi(u)^2 / (1 - Phi(u)); its stationary point satisfies
 * 2u (1 - Phi(u)) = phi(u), whose root is ORC_GAUSS_U = 0.61200318...  With
 * sigma estimated by maximum likelihood, rms(w) (Sec. 3.1):
 * Delta = fp32(ORC_GAUSS_U * sqrt(sum w^2 / n)) (fp64 sum in index order),
 * kept set {i : |w_i| > Delta} in fp32, alpha = fp32(mean of the kept
 * magnitudes) as in Eq. (5).
 */
static int ternarize_gauss(const float* w, int64_t n, int64_t stride, int8_t* t,
                           int64_t tstride, float* alpha, float* delta) {
  double Q = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    const double v = (double)w[i * stride];
    Q = Q + v * v;
  }
  float d = (float)(ORC_GAUSS_U * sqrt(Q / (double)n));
  double K = 0.0;
  int64_t cnt = 0;
  for (int64_t i = 0; i < n; ++i) {
    float a = fabsf(w[i * stride]);
    if (a > d) {
      K = K + (double)a;
      cnt += 1;
      t[i * tstride] = (int8_t)sign_of(w[i * stride]);
    } else {
      t[i * tstride] = 0;
    }
  }
  *alpha = cnt > 0 ? (float)(K / (double)cnt) : 0.0f;
  *delta = d;
  return ORC_OK;
}

int orc_ternarize_group(const float* w, int64_t n, int64_t stride, int method,
                        int8_t* t, int64_t tstride, float* alpha, float* delta) {
  if (!w || !t || !alpha || !delta) return ORC_ERR_NULL;
  if (n < 1) return ORC_ERR_SHAPE;
  for (int64_t i = 0; i < n; ++i)
    if (!isfinite(w[i * stride])) return ORC_ERR_NONFINITE;
  if (method == ORC_TERN_EXACT)
    return ternarize_exact(w, n, stride, t, tstride, alpha, delta);
  if (method == ORC_TERN_EXP_LEMMA)
    return ternarize_lemma(w, n, stride, t, tstride, alpha, delta);
  if (method == ORC_TERN_GAUSS)
    return ternarize_gauss(w, n, stride, t, tstride, alpha, delta);
  return ORC_ERR_SHAPE;
}

/*
 * Eq. (3)-(4): one threshold for the positive weights, I+ = {i : w_i > Dp},
 * one for the negative ones, I- = {i : w_i < -Dn}, and one scale.  Eq. (4)
 * gives alpha = (sum_{I+}|w| + sum_{I-}|w|) / (|I+| + |I-|) and the
 * thresholds maximising the square of that sum over |I+| + |I-|.  Every
 * distinct pair of kept sets is a pair of prefixes of the positive and of
 * the negative magnitudes, each sorted in decreasing order (ties by
 * position), so the exhaustive search visits every pair (a, b), 0 <= a <= n+,
 * 0 <= b <= n-, a + b >= 1: P_a and N_b are fp64 prefix sums in sorted
 * order, T = P_a + N_b, f = T*T / (a + b), and the first maximum in the
 * order (a, then b) with a strict > is kept.  alpha = fp32(T / (a + b));
 * Dp = the (a+1)-th positive magnitude (0 if all positives are kept), Dn
 * likewise; t = +1 on the a largest positives, -1 on the b largest negatives.
 * Zeros are in neither set.  No group has a zero f maximum unless it is all
 * zeros (then alpha = Dp = Dn = 0, all codes 0).
 */
int orc_ternarize_group_asym(const float* w, int64_t n, int64_t stride, int8_t* t,
                             int64_t tstride, float* alpha, float* delta_p, float* delta_n) {
  if (!w || !t || !alpha || !delta_p || !delta_n) return ORC_ERR_NULL;
  if (n < 1) return ORC_ERR_SHAPE;
  for (int64_t i = 0; i < n; ++i)
    if (!isfinite(w[i * stride])) return ORC_ERR_NONFINITE;
  mag_t* pos = (mag_t*)malloc(sizeof(mag_t) * (size_t)n);
  mag_t* neg = (mag_t*)malloc(sizeof(mag_t) * (size_t)n);
  double* P = (double*)malloc(sizeof(double) * (size_t)(n + 1));
  double* N = (double*)malloc(sizeof(double) * (size_t)(n + 1));
  if (!pos || !neg || !P || !N) {
    free(pos); free(neg); free(P); free(N);
    return ORC_ERR_SHAPE;
  }
  int64_t np = 0, nn = 0;
  for (int64_t i = 0; i < n; ++i) {
    const float v = w[i * stride];
    if (v > 0.0f) { pos[np].a = v; pos[np].idx = i; ++np; }
    if (v < 0.0f) { neg[nn].a = -v; neg[nn].idx = i; ++nn; }
  }
  qsort(pos, (size_t)np, sizeof(mag_t), cmp_mag);
  qsort(neg, (size_t)nn, sizeof(mag_t), cmp_mag);
  P[0] = 0.0;
  for (int64_t a = 1; a <= np; ++a) P[a] = P[a - 1] + (double)pos[a - 1].a;
  N[0] = 0.0;
  for (int64_t b = 1; b <= nn; ++b) N[b] = N[b - 1] + (double)neg[b - 1].a;
  double bestf = 0.0, bestT = 0.0;
  int64_t ba = 0, bb = 0;
  for (int64_t a = 0; a <= np; ++a)
    for (int64_t b = 0; b <= nn; ++b) {
      if (a + b == 0) continue;
      const double T = P[a] + N[b];
      const double f = (T * T) / (double)(a + b);
      if (f > bestf) {
        bestf = f;
        bestT = T;
        ba = a;
        bb = b;
      }
    }
  *alpha = ba + bb > 0 ? (float)(bestT / (double)(ba + bb)) : 0.0f;
  *delta_p = ba < np ? pos[ba].a : 0.0f;
  *delta_n = bb < nn ? neg[bb].a : 0.0f;
  for (int64_t i = 0; i < n; ++i) t[i * tstride] = 0;
  for (int64_t a = 0; a < ba; ++a) t[pos[a].idx * tstride] = 1;
  for (int64_t b = 0; b < bb; ++b) t[neg[b].idx * tstride] = -1;
  free(pos); free(neg); free(P); free(N);
  return ORC_OK;
}

static int cmp_float_up(const void* pa, const void* pb) {
  const float x = *(const float*)pa, y = *(const float*)pb;
  return x < y ? -1 : (x > y ? 1 : 0);
}

/*
 * Sec. 3.1: the Kolmogorov-Smirnov distance of the weight magnitudes to the
 * two reference laws, each fitted by maximum likelihood: the half-normal law
 * of N(0, sigma), sigma = rms(W), CDF erf(x / (sigma sqrt 2)); and the
 * exponential law of scale mu = mean|W| (the 1/lambda of Lemma 1), CDF
 * 1 - exp(-x / mu).  Computed on at most ORC_KS_SAMPLE magnitudes: every s-th
 * weight in storage order, s = ceil(n / ORC_KS_SAMPLE).  With the sample
 * sorted ascending, m_(1) <= ... <= m_(ns): sigma^2 = sum m^2 / ns and
 * mu = sum m / ns (fp64, ascending order), and
 * D = max_i max(i/ns - F(m_(i)), F(m_(i)) - (i-1)/ns).  A sample of zeros
 * gives D = 0 for both.  d[0] = D for the half-normal law, d[1] for the
 * exponential one.
 */
int orc_ks_distances(const float* w, int64_t n, double* d) {
  if (!w || !d) return ORC_ERR_NULL;
  if (n < 1) return ORC_ERR_SHAPE;
  for (int64_t i = 0; i < n; ++i)
    if (!isfinite(w[i])) return ORC_ERR_NONFINITE;
  const int64_t step = (n + ORC_KS_SAMPLE - 1) / ORC_KS_SAMPLE;
  const int64_t ns = (n + step - 1) / step;
  float* m = (float*)malloc(sizeof(float) * (size_t)ns);
  if (!m) return ORC_ERR_SHAPE;
  for (int64_t j = 0; j < ns; ++j) m[j] = fabsf(w[j * step]);
  qsort(m, (size_t)ns, sizeof(float), cmp_float_up);
  double Q = 0.0, S = 0.0;
  for (int64_t j = 0; j < ns; ++j) {
    const double v = (double)m[j];
    Q = Q + v * v;
    S = S + v;
  }
  const double sigma = sqrt(Q / (double)ns), mu = S / (double)ns;
  double dg = 0.0, de = 0.0;
  if (mu > 0.0) {
    for (int64_t j = 0; j < ns; ++j) {
      const double x = (double)m[j];
      const double hi = (double)(j + 1) / (double)ns, lo = (double)j / (double)ns;
      const double fg = erf(x / (sigma * sqrt(2.0)));
      const double fe = 1.0 - exp(-x / mu);
      dg = fmax(dg, fmax(hi - fg, fg - lo));
      de = fmax(de, fmax(hi - fe, fe - lo));
    }
  }
  d[0] = dg;
  d[1] = de;
  free(m);
  return ORC_OK;
}

/*
 * Sec. 3.2 / Fig. 2: a group is G consecutive input channels of one filter at
 * one tap (o, r, s); the layer is solved as K/G independent sub-problems
 * (Eq. (2)).  Input weights [O][C][R][S]; codes written [O][R][S][C].
 */
int orc_ternarize(const float* w, int64_t O, int64_t C, int32_t R, int32_t S,
                  int32_t G, int32_t method, int8_t* t, float* alpha,
                  float* delta) {
  if (!w || !t || !alpha || !delta) return ORC_ERR_NULL;
  if (O < 1 || C < 1 || R < 1 || S < 1) return ORC_ERR_SHAPE;
  if (G < 1 || C % G != 0) return ORC_ERR_GROUP;
  const int64_t K = (int64_t)R * S * C;
  const int64_t ng = K / G;
  for (int64_t i = 0; i < O * K; ++i)
    if (!isfinite(w[i])) return ORC_ERR_NONFINITE;
  if (method == ORC_TERN_KS) {
    /* Sec. 3.1: the K-S test picks the reference law of the layer, and each
     * group takes that law's threshold: exponential -> Lemma 1, Gaussian ->
     * ORC_GAUSS_U * rms (the exponential law only when strictly closer). */
    double d[2];
    int rc = orc_ks_distances(w, O * K, d);
    if (rc != ORC_OK) return rc;
    method = d[1] < d[0] ? ORC_TERN_EXP_LEMMA : ORC_TERN_GAUSS;
  }
  for (int64_t o = 0; o < O; ++o)
    for (int32_t r = 0; r < R; ++r)
      for (int32_t s = 0; s < S; ++s)
        for (int64_t cb = 0; cb < C / G; ++cb) {
          /* w[o][c][r][s], c = cb*G + ci: stride between channels is R*S */
          const float* src = w + ((o * C + cb * G) * R + r) * S + s;
          const int64_t k0 = ((int64_t)r * S + s) * C + cb * G;
          const int64_t g = k0 / G;
          int rc = orc_ternarize_group(src, G, (int64_t)R * S, method,
                                       t + o * K + k0, 1, alpha + o * ng + g,
                                       delta + o * ng + g);
          if (rc != ORC_OK) return rc;
        }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* 2-bit code storage                                                        */
/* ------------------------------------------------------------------------ */

void orc_pack_codes(const int8_t* t, int64_t O, int64_t K, uint8_t* codes) {
  const int64_t rb = (K + 3) / 4;
  for (int64_t o = 0; o < O; ++o)
    for (int64_t b = 0; b < rb; ++b) {
      unsigned byte = 0;
      for (int q = 0; q < 4; ++q) {
        int64_t k = 4 * b + q;
        unsigned c = 0;
        if (k < K) {
          int8_t v = t[o * K + k];
          c = v == 1 ? 1u : (v == -1 ? 3u : 0u);
        }
        byte |= c << (2 * q);
      }
      codes[o * rb + b] = (uint8_t)byte;
    }
}

void orc_unpack_codes(const uint8_t* codes, int64_t O, int64_t K, int8_t* t) {
  const int64_t rb = (K + 3) / 4;
  for (int64_t o = 0; o < O; ++o)
    for (int64_t k = 0; k < K; ++k) {
      unsigned c = (codes[o * rb + k / 4] >> (2 * (k % 4))) & 3u;
      t[o * K + k] = c == 1 ? 1 : (c == 3 ? -1 : 0);
    }
}

/* ------------------------------------------------------------------------ */
/* Activation quantization (Sec. 4: activations quantized to 8 or 4 bits     */
/* before each convolution; one scale per tensor)                            */
/* ------------------------------------------------------------------------ */

int orc_quantize_act(const float* x, int64_t n, int32_t bits,
                     const float* scale_in, uint8_t* q, float* scale_out) {
  if (!x || !q || !scale_out) return ORC_ERR_NULL;
  if (bits != 8 && bits != 4) return ORC_ERR_BITS;
  if (n < 0) return ORC_ERR_SHAPE;
  if (bits == 4 && (n % 2) != 0) return ORC_ERR_BITS;
  const float qmax = bits == 8 ? 255.0f : 15.0f;
  float s;
  if (scale_in) {
    s = *scale_in;
  } else {
    float mx = 0.0f;
    for (int64_t i = 0; i < n; ++i)
      if (x[i] > mx) mx = x[i]; /* NaN never compares greater */
    s = mx > 0.0f ? mx / qmax : 1.0f;
  }
  *scale_out = s;
  for (int64_t i = 0; i < n; ++i) {
    float v = rintf(x[i] / s);       /* IEEE division, round half to even */
    v = fminf(fmaxf(v, 0.0f), qmax); /* NaN -> 0, negative -> 0 */
    unsigned u = (unsigned)v;
    if (bits == 8) {
      q[i] = (uint8_t)u;
    } else if (i % 2 == 0) {
      q[i / 2] = (uint8_t)u;
    } else {
      q[i / 2] = (uint8_t)(q[i / 2] | (u << 4));
    }
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Layer: implicit-GEMM convolution and GEMM                                 */
/* ------------------------------------------------------------------------ */

static unsigned act_at(const uint8_t* q, int32_t bits, int64_t e) {
  if (bits == 8) return q[e];
  return (q[e / 2] >> (4 * (e % 2))) & 15u;
}

typedef struct {
  int64_t B, H, W, C, O, Ho, Wo, K;
  int32_t R, S, sh, sw, ph, pw;
} geom_t;

static int conv_geom(int64_t B, int64_t H, int64_t W, int64_t C, int64_t O,
                     int32_t R, int32_t S, int32_t sh, int32_t sw, int32_t ph,
                     int32_t pw, geom_t* g) {
  if (B < 1 || H < 1 || W < 1 || C < 1 || O < 1 || R < 1 || S < 1 || sh < 1 ||
      sw < 1 || ph < 0 || pw < 0)
    return ORC_ERR_SHAPE;
  if (H + 2 * ph < R || W + 2 * pw < S) return ORC_ERR_SHAPE;
  g->B = B; g->H = H; g->W = W; g->C = C; g->O = O;
  g->R = R; g->S = S; g->sh = sh; g->sw = sw; g->ph = ph; g->pw = pw;
  g->Ho = (H + 2 * ph - R) / sh + 1;
  g->Wo = (W + 2 * pw - S) / sw + 1;
  g->K = (int64_t)R * S * C;
  return ORC_OK;
}

/* A[m][k] of the implicit GEMM: the input pixel under tap (r, s) for output
 * pixel m = (b, ho, wo), channel c; 0 outside the image (zero padding). */
static unsigned conv_a(const uint8_t* q, int32_t bits, const geom_t* g,
                       int64_t m, int64_t k) {
  int64_t wo = m % g->Wo;
  int64_t ho = (m / g->Wo) % g->Ho;
  int64_t b = m / (g->Wo * g->Ho);
  int64_t c = k % g->C;
  int64_t rs = k / g->C;
  int64_t s = rs % g->S;
  int64_t r = rs / g->S;
  int64_t hi = ho * g->sh - g->ph + r;
  int64_t wi = wo * g->sw - g->pw + s;
  if (hi < 0 || hi >= g->H || wi < 0 || wi >= g->W) return 0;
  return act_at(q, bits, ((b * g->H + hi) * g->W + wi) * g->C + c);
}

int orc_group_sums_conv(const uint8_t* q, int32_t bits, int64_t B, int64_t H,
                        int64_t W, int64_t C, const uint8_t* codes, int64_t O,
                        int32_t R, int32_t S, int32_t sh, int32_t sw,
                        int32_t ph, int32_t pw, int32_t G, int64_t row0,
                        int64_t nrows, int32_t* P) {
  if (!q || !codes || !P) return ORC_ERR_NULL;
  if (bits != 8 && bits != 4) return ORC_ERR_BITS;
  geom_t g;
  int rc = conv_geom(B, H, W, C, O, R, S, sh, sw, ph, pw, &g);
  if (rc) return rc;
  if (G < 1 || C % G != 0) return ORC_ERR_GROUP;
  const int64_t M = g.B * g.Ho * g.Wo;
  if (row0 < 0 || nrows < 0 || row0 + nrows > M) return ORC_ERR_SHAPE;
  const int64_t K = g.K, ng = K / G;
  int8_t* t = (int8_t*)malloc((size_t)(O * K));
  if (!t) return ORC_ERR_SHAPE;
  orc_unpack_codes(codes, O, K, t);
  for (int64_t i = 0; i < nrows; ++i) {
    int64_t m = row0 + i;
    for (int64_t o = 0; o < O; ++o)
      for (int64_t gi = 0; gi < ng; ++gi) {
        int64_t acc = 0;
        for (int64_t k = gi * G; k < (gi + 1) * G; ++k)
          acc += (int64_t)t[o * K + k] * (int64_t)conv_a(q, bits, &g, m, k);
        P[(i * O + o) * ng + gi] = (int32_t)acc;
      }
  }
  free(t);
  return ORC_OK;
}

int orc_conv2d(const uint8_t* q, int32_t bits, float sx, int64_t B, int64_t H,
               int64_t W, int64_t C, const uint8_t* codes, const float* alpha,
               int64_t O, int32_t R, int32_t S, int32_t sh, int32_t sw,
               int32_t ph, int32_t pw, int32_t G, int64_t row0, int64_t nrows,
               int32_t nthreads, float* y) {
  if (!q || !codes || !alpha || !y) return ORC_ERR_NULL;
  if (bits != 8 && bits != 4) return ORC_ERR_BITS;
  geom_t g;
  int rc = conv_geom(B, H, W, C, O, R, S, sh, sw, ph, pw, &g);
  if (rc) return rc;
  if (G < 1 || C % G != 0) return ORC_ERR_GROUP;
  const int64_t M = g.B * g.Ho * g.Wo;
  if (nrows < 0) {
    row0 = 0;
    nrows = M;
  }
  if (row0 < 0 || row0 + nrows > M) return ORC_ERR_SHAPE;
  const int64_t K = g.K, ng = K / G;
  int8_t* t = (int8_t*)malloc((size_t)(O * K));
  if (!t) return ORC_ERR_SHAPE;
  orc_unpack_codes(codes, O, K, t);
  const int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 16) num_threads(nt)
  for (int64_t m = row0; m < row0 + nrows; ++m) {
    for (int64_t o = 0; o < O; ++o) {
      double acc = 0.0;
      for (int64_t gi = 0; gi < ng; ++gi) {
        int64_t P = 0;
        for (int64_t k = gi * G; k < (gi + 1) * G; ++k)
          P += (int64_t)t[o * K + k] * (int64_t)conv_a(q, bits, &g, m, k);
        acc += (double)alpha[o * ng + gi] * (double)P;
      }
      y[m * O + o] = (float)((double)sx * acc);
    }
  }
  free(t);
  return ORC_OK;
}

int orc_conv2d_rows(const uint8_t* q, int32_t bits, float sx, int64_t B, int64_t H,
                    int64_t W, int64_t C, const uint8_t* codes, const float* alpha,
                    int64_t O, int32_t R, int32_t S, int32_t sh, int32_t sw,
                    int32_t ph, int32_t pw, int32_t G, const int64_t* rows,
                    int64_t nrows, int32_t nthreads, float* y, double* mag) {
  if (!q || !codes || !alpha || !rows || !y || !mag) return ORC_ERR_NULL;
  if (bits != 8 && bits != 4) return ORC_ERR_BITS;
  geom_t g;
  int rc = conv_geom(B, H, W, C, O, R, S, sh, sw, ph, pw, &g);
  if (rc) return rc;
  if (G < 1 || C % G != 0) return ORC_ERR_GROUP;
  const int64_t M = g.B * g.Ho * g.Wo;
  for (int64_t i = 0; i < nrows; ++i)
    if (rows[i] < 0 || rows[i] >= M) return ORC_ERR_SHAPE;
  const int64_t K = g.K, ng = K / G;
  int8_t* t = (int8_t*)malloc((size_t)(O * K));
  if (!t) return ORC_ERR_SHAPE;
  orc_unpack_codes(codes, O, K, t);
  const int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 4) num_threads(nt)
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t m = rows[i];
    for (int64_t o = 0; o < O; ++o) {
      double acc = 0.0, abs_acc = 0.0;
      for (int64_t gi = 0; gi < ng; ++gi) {
        int64_t P = 0;
        for (int64_t k = gi * G; k < (gi + 1) * G; ++k)
          P += (int64_t)t[o * K + k] * (int64_t)conv_a(q, bits, &g, m, k);
        acc += (double)alpha[o * ng + gi] * (double)P;
        abs_acc += (double)alpha[o * ng + gi] * (double)(P < 0 ? -P : P);
      }
      y[i * O + o] = (float)((double)sx * acc);
      mag[i * O + o] = (double)sx * abs_acc;
    }
  }
  free(t);
  return ORC_OK;
}

int orc_gemm(const uint8_t* q, int32_t bits, float sx, int64_t M, int64_t K,
             const uint8_t* codes, const float* alpha, int64_t O, int32_t G,
             int32_t nthreads, float* y) {
  if (!q || !codes || !alpha || !y) return ORC_ERR_NULL;
  if (bits != 8 && bits != 4) return ORC_ERR_BITS;
  if (M < 1 || K < 1 || O < 1) return ORC_ERR_SHAPE;
  if (G < 1 || K % G != 0) return ORC_ERR_GROUP;
  const int64_t ng = K / G;
  int8_t* t = (int8_t*)malloc((size_t)(O * K));
  if (!t) return ORC_ERR_SHAPE;
  orc_unpack_codes(codes, O, K, t);
  const int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 16) num_threads(nt)
  for (int64_t m = 0; m < M; ++m) {
    for (int64_t o = 0; o < O; ++o) {
      double acc = 0.0;
      for (int64_t gi = 0; gi < ng; ++gi) {
        int64_t P = 0;
        for (int64_t k = gi * G; k < (gi + 1) * G; ++k)
          P += (int64_t)t[o * K + k] * (int64_t)act_at(q, bits, m * K + k);
        acc += (double)alpha[o * ng + gi] * (double)P;
      }
      y[m * O + o] = (float)((double)sx * acc);
    }
  }
  free(t);
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Fixed-point group scales (Sec. 4)                                          */
/* ------------------------------------------------------------------------ */

int orc_dfp_alpha(const float* alpha, int64_t n, int32_t bits, int8_t* A,
                  int32_t* fl) {
  if (!alpha || !A || !fl) return ORC_ERR_NULL;
  if (bits != 8 && bits != 4) return ORC_ERR_BITS;
  if (n < 0) return ORC_ERR_SHAPE;
  double amax = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    if (!isfinite(alpha[i]) || alpha[i] < 0.0f) return ORC_ERR_NONFINITE;
    if (alpha[i] > amax) amax = alpha[i];
  }
  int32_t f = 0;
  if (amax > 0.0) {
    /* amax = m 2^e with m in [0.5, 1): log2(amax) lies in [e-1, e), and
     * equals e-1 only when m = 0.5 */
    int e;
    double m = frexp(amax, &e);
    int ceil_log2 = (m == 0.5) ? e - 1 : e;
    f = bits - (ceil_log2 + 1);
  }
  const double amax_code = (double)((1 << (bits - 1)) - 1);
  for (int64_t i = 0; i < n; ++i) {
    double v = amax > 0.0 ? nearbyint(ldexp((double)alpha[i], f)) : 0.0;
    if (v > amax_code) v = amax_code;
    A[i] = (int8_t)v;
  }
  *fl = f;
  return ORC_OK;
}

int orc_conv2d_dfp(const uint8_t* q, int32_t bits, float sx, int64_t B,
                   int64_t H, int64_t W, int64_t C, const uint8_t* codes,
                   const int8_t* A, int32_t fl, int64_t O, int32_t R,
                   int32_t S, int32_t sh, int32_t sw, int32_t ph, int32_t pw,
                   int32_t G, int64_t row0, int64_t nrows, int32_t nthreads,
                   float* y) {
  if (!q || !codes || !A || !y) return ORC_ERR_NULL;
  if (bits != 8 && bits != 4) return ORC_ERR_BITS;
  geom_t g;
  int rc = conv_geom(B, H, W, C, O, R, S, sh, sw, ph, pw, &g);
  if (rc) return rc;
  if (G < 1 || C % G != 0) return ORC_ERR_GROUP;
  const int64_t M = g.B * g.Ho * g.Wo;
  if (nrows < 0) {
    row0 = 0;
    nrows = M;
  }
  if (row0 < 0 || row0 + nrows > M) return ORC_ERR_SHAPE;
  const int64_t K = g.K, ng = K / G;
  int8_t* t = (int8_t*)malloc((size_t)(O * K));
  if (!t) return ORC_ERR_SHAPE;
  orc_unpack_codes(codes, O, K, t);
  const double scale = (double)sx * ldexp(1.0, -fl);
  const int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 16) num_threads(nt)
  for (int64_t m = row0; m < row0 + nrows; ++m) {
    for (int64_t o = 0; o < O; ++o) {
      int64_t acc = 0;
      for (int64_t k = 0; k < K; ++k)
        acc += (int64_t)A[o * ng + k / G] * (int64_t)t[o * K + k] *
               (int64_t)conv_a(q, bits, &g, m, k);
      y[m * O + o] = (float)((double)acc * scale);
    }
  }
  free(t);
  return ORC_OK;
}

int orc_gemm_dfp(const uint8_t* q, int32_t bits, float sx, int64_t M,
                 int64_t K, const uint8_t* codes, const int8_t* A, int32_t fl,
                 int64_t O, int32_t G, int32_t nthreads, float* y) {
  if (!q || !codes || !A || !y) return ORC_ERR_NULL;
  if (bits != 8 && bits != 4) return ORC_ERR_BITS;
  if (M < 1 || K < 1 || O < 1) return ORC_ERR_SHAPE;
  if (G < 1 || K % G != 0) return ORC_ERR_GROUP;
  const int64_t ng = K / G;
  int8_t* t = (int8_t*)malloc((size_t)(O * K));
  if (!t) return ORC_ERR_SHAPE;
  orc_unpack_codes(codes, O, K, t);
  const double scale = (double)sx * ldexp(1.0, -fl);
  const int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 16) num_threads(nt)
  for (int64_t m = 0; m < M; ++m) {
    for (int64_t o = 0; o < O; ++o) {
      int64_t acc = 0;
      for (int64_t k = 0; k < K; ++k)
        acc += (int64_t)A[o * ng + k / G] * (int64_t)t[o * K + k] *
               (int64_t)act_at(q, bits, m * K + k);
      y[m * O + o] = (float)((double)acc * scale);
    }
  }
  free(t);
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* First layer at 8-bit weights (Sec. 4, 8w-8a)                               */
/* ------------------------------------------------------------------------ */

int orc_w8_quantize(const float* w, int64_t n, int8_t* W8, int32_t* fl) {
  if (!w || !W8 || !fl) return ORC_ERR_NULL;
  if (n < 0) return ORC_ERR_SHAPE;
  double wmax = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    if (!isfinite(w[i])) return ORC_ERR_NONFINITE;
    double a = fabs((double)w[i]);
    if (a > wmax) wmax = a;
  }
  int32_t f = 0;
  if (wmax > 0.0) {
    int e;
    double m = frexp(wmax, &e); /* wmax = m 2^e, m in [0.5, 1) */
    int ceil_log2 = (m == 0.5) ? e - 1 : e;
    f = 8 - (ceil_log2 + 1);
  }
  for (int64_t i = 0; i < n; ++i) {
    double v = wmax > 0.0 ? nearbyint(ldexp((double)w[i], f)) : 0.0;
    if (v > 127.0) v = 127.0;
    if (v < -128.0) v = -128.0;
    W8[i] = (int8_t)v;
  }
  *fl = f;
  return ORC_OK;
}

int orc_conv2d_w8(const uint8_t* q, int32_t bits, float sx, int64_t B,
                  int64_t H, int64_t W, int64_t C, const int8_t* W8,
                  int32_t fl, int64_t O, int32_t R, int32_t S, int32_t sh,
                  int32_t sw, int32_t ph, int32_t pw, int64_t row0,
                  int64_t nrows, int32_t nthreads, float* y) {
  if (!q || !W8 || !y) return ORC_ERR_NULL;
  if (bits != 8 && bits != 4) return ORC_ERR_BITS;
  geom_t g;
  int rc = conv_geom(B, H, W, C, O, R, S, sh, sw, ph, pw, &g);
  if (rc) return rc;
  const int64_t M = g.B * g.Ho * g.Wo;
  if (nrows < 0) {
    row0 = 0;
    nrows = M;
  }
  if (row0 < 0 || row0 + nrows > M) return ORC_ERR_SHAPE;
  const double scale = (double)sx * ldexp(1.0, -fl);
  const int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 16) num_threads(nt)
  for (int64_t m = row0; m < row0 + nrows; ++m) {
    for (int64_t o = 0; o < O; ++o) {
      int64_t acc = 0;
      for (int64_t c = 0; c < C; ++c)
        for (int32_t r = 0; r < R; ++r)
          for (int32_t s = 0; s < S; ++s)
            acc += (int64_t)W8[((o * C + c) * R + r) * S + s] *
                   (int64_t)conv_a(q, bits, &g, m, ((int64_t)r * S + s) * C + c);
      y[m * O + o] = (float)((double)acc * scale);
    }
  }
  return ORC_OK;
}

int orc_max_threads(void) { return omp_get_max_threads(); }

double orc_gauss_u(void) { return ORC_GAUSS_U; }

/*
 * Eq. (3)-(4) per group over a layer, grouped as orc_ternarize does.
 */
int orc_ternarize_asym(const float* w, int64_t O, int64_t C, int32_t R, int32_t S,
                       int32_t G, int8_t* t, float* alpha, float* delta_p, float* delta_n) {
  if (!w || !t || !alpha || !delta_p || !delta_n) return ORC_ERR_NULL;
  if (O < 1 || C < 1 || R < 1 || S < 1) return ORC_ERR_SHAPE;
  if (G < 1 || C % G != 0) return ORC_ERR_GROUP;
  const int64_t K = (int64_t)R * S * C;
  const int64_t ng = K / G;
  for (int64_t o = 0; o < O; ++o)
    for (int32_t r = 0; r < R; ++r)
      for (int32_t s = 0; s < S; ++s)
        for (int64_t cb = 0; cb < C / G; ++cb) {
          const float* src = w + ((o * C + cb * G) * R + r) * S + s;
          const int64_t k0 = ((int64_t)r * S + s) * C + cb * G;
          const int64_t g = k0 / G;
          int rc = orc_ternarize_group_asym(src, G, (int64_t)R * S, t + o * K + k0, 1,
                                            alpha + o * ng + g, delta_p + o * ng + g,
                                            delta_n + o * ng + g);
          if (rc != ORC_OK) return rc;
        }
  return ORC_OK;
}
