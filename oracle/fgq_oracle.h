/*
 * fgq_oracle.h -- plain CPU oracle for Fine-Grained Quantization (FGQ)
 * inference (Mellempudi et al., "Ternary Neural Networks with Fine-Grained
 * Quantization", arXiv 1705.01462).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link or
 * call this code; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark use it.  It shares no code, header, table or helper with the
 * HIP library.
 *
 * What it computes, each function citing the passage it follows:
 *   orc_ternarize     Sec. 3 threshold rule + Eq. (1) objective, solved per
 *                     group (Sec. 3.1, Eq. (2)) with the symmetric closed form
 *                     of Eq. (5) by exhaustive search over the thresholds
 *                     (the "brute-force" solve of Sec. 3.1 / Sec. 4); groups
 *                     are N consecutive input channels at a fixed filter tap
 *                     (Sec. 3.2, Fig. 2).  Method 1 is Lemma 1 (Delta = mean|W|);
 *                     method 3 the Gaussian-optimal threshold 0.612 rms(W);
 *                     method 4 picks 1 or 3 per layer by the K-S test (Sec. 3.1).
 *   orc_ternarize_asym  Eq. (3)-(4): positive and negative thresholds, one
 *                     scale, solved exhaustively.
 *   orc_ks_distances  the K-S distances behind method 4.
 *   orc_pack_codes    2-bit storage of ternary codes (4 per byte).
 *   orc_quantize_act  activations quantized to 8 or 4 bits with one scale per
 *                     tensor (Sec. 4, experimental setup).
 *   orc_group_sums    exact integer partial sums P_g = sum_{i in g} t_i q_i
 *                     (Sec. 4: 32-bit accumulation).
 *   orc_conv2d        y = s_x * sum_g alpha_g * P_g for an implicit-GEMM conv
 *   orc_gemm          (Sec. 3.1 Eq. (2) applied to a layer; one multiply per
 *                     group, Sec. 4 Discussion).
 *   orc_dfp_alpha     the group scales quantized to an 8- or 4-bit dynamic
 *                     fixed point with one exponent per layer (Sec. 4,
 *                     experimental setup).
 *   orc_conv2d_dfp    the layer with those scales: an exact integer sum of
 *   orc_gemm_dfp      (A_g t_k) q_k and one scaling by s_x 2^-fl (Sec. 4).
 *   orc_w8_quantize   the first layer kept at 8-bit weights (Sec. 4, 8w-8a):
 *   orc_conv2d_w8     weights as an 8-bit dynamic fixed point, one exponent
 *                     per layer, and that layer computed the same way.
 *
 * Parity status: ternarize, quantize, group sums, conv2d and gemm are pinned
 * by the tests (brute-force enumeration, Lemma 1 statistics, closed forms,
 * reduction to a library convolution); the variants (asymmetric thresholds,
 * Gaussian threshold, K-S distances and choice) by enumeration, the Eq. (5)
 * optimum, a root found by scipy, scipy's K-S statistic and large-sample
 * limits; see tests/test_oracle_*.py.
 *
 * Conventions (shared with the library only by specification, not by code):
 *   weights   fp32 [O][C][R][S]
 *   codes     2-bit, reduction index k = (r*S + s)*C + c, row o holds
 *             ceil(K/4) bytes; element k sits in bits [2(k%4), 2(k%4)+1] of
 *             byte k/4; 00 -> 0, 01 -> +1, 11 -> -1 (10 never written)
 *   alpha     fp32 [O][K/G], group g = k / G (fixed point: int8 A [O][K/G]
 *             and one fractional length fl per layer)
 *   acts      NHWC, u8 one per byte or u4 two per byte (even element in the
 *             low nibble)
 *   output    fp32 NHWC [B][Ho][Wo][O] (GEMM: [M][O])
 */
#ifndef FGQ_ORACLE_H
#define FGQ_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  ORC_OK = 0,
  ORC_ERR_NULL = 1,
  ORC_ERR_SHAPE = 2,
  ORC_ERR_GROUP = 3,
  ORC_ERR_BITS = 4,
  ORC_ERR_NONFINITE = 5
};

enum { ORC_TERN_EXACT = 0, ORC_TERN_EXP_LEMMA = 1, ORC_TERN_GAUSS = 3, ORC_TERN_KS = 4 };

/* Root of 2u(1 - Phi(u)) = phi(u): the Gaussian-optimal threshold of Eq. (5)
 * in units of sigma (see orc_ternarize_group, method ORC_TERN_GAUSS). */
#define ORC_GAUSS_U 0.61200318096248076
/* Sample size of the K-S distances (orc_ks_distances). */
#define ORC_KS_SAMPLE 16384

/* One group of n weights read at w[i*stride].  Writes t[i*tstride] in
 * {-1,0,1}, *alpha, *delta.  Returns ORC_ERR_NONFINITE on NaN/Inf. */
int orc_ternarize_group(const float* w, int64_t n, int64_t stride, int method,
                        int8_t* t, int64_t tstride, float* alpha, float* delta);

/* Whole layer.  t is [O][R][S][C] (unpacked codes), alpha/delta [O][K/G]. */
/* Eq. (3)-(4): asymmetric thresholds Dp, Dn with one alpha, exhaustive over
 * pairs of prefixes; t in {-1,0,1}.  Returns ORC_ERR_NONFINITE on NaN/Inf. */
int orc_ternarize_group_asym(const float* w, int64_t n, int64_t stride, int8_t* t,
                             int64_t tstride, float* alpha, float* delta_p, float* delta_n);
int orc_ternarize_asym(const float* w, int64_t O, int64_t C, int32_t R, int32_t S,
                       int32_t G, int8_t* t, float* alpha, float* delta_p, float* delta_n);
/* Sec. 3.1 K-S goodness of fit of |w| (n values, storage order) against the
 * half-normal (d[0]) and exponential (d[1]) laws fitted by maximum likelihood. */
int orc_ks_distances(const float* w, int64_t n, double* d);
/* ORC_GAUSS_U, for the tests. */
double orc_gauss_u(void);
int orc_ternarize(const float* w, int64_t O, int64_t C, int32_t R, int32_t S,
                  int32_t G, int32_t method, int8_t* t, float* alpha,
                  float* delta);

/* 2-bit packing / unpacking of an [O][K] code matrix. */
void orc_pack_codes(const int8_t* t, int64_t O, int64_t K, uint8_t* codes);
void orc_unpack_codes(const uint8_t* codes, int64_t O, int64_t K, int8_t* t);

/* Quantize n fp32 values to bits (8|4).  scale_in may be NULL (dynamic
 * scale s = max(max x, 0)/qmax, or 1 if that is 0).  q holds n bytes (bits=8)
 * or n/2 bytes (bits=4, n even).  *scale_out receives s. */
int orc_quantize_act(const float* x, int64_t n, int32_t bits,
                     const float* scale_in, uint8_t* q, float* scale_out);

/* Exact group sums for output rows [row0, row0+nrows) of a conv:
 * P[(row-row0)][o][g], int32. */
int orc_group_sums_conv(const uint8_t* q, int32_t bits, int64_t B, int64_t H,
                        int64_t W, int64_t C, const uint8_t* codes, int64_t O,
                        int32_t R, int32_t S, int32_t sh, int32_t sw,
                        int32_t ph, int32_t pw, int32_t G, int64_t row0,
                        int64_t nrows, int32_t* P);

/* y[m][o] = fp32( s_x * sum_g alpha[o][g] * P[m][o][g] ), fp64 sum.
 * Rows [row0, row0+nrows) only (nrows < 0: all rows); y is indexed by the
 * absolute row.  nthreads <= 0: OpenMP default. */
int orc_conv2d(const uint8_t* q, int32_t bits, float sx, int64_t B, int64_t H,
               int64_t W, int64_t C, const uint8_t* codes, const float* alpha,
               int64_t O, int32_t R, int32_t S, int32_t sh, int32_t sw,
               int32_t ph, int32_t pw, int32_t G, int64_t row0, int64_t nrows,
               int32_t nthreads, float* y);

/* The layer of orc_conv2d on a list of output rows (rows[0..nrows), any
 * order): y[i][o] is orc_conv2d's value for row rows[i], and mag[i][o] =
 * s_x * sum_g alpha[o][g] * |P_g| (fp64), the summand magnitude against
 * which the matrix-core kernels' tolerance is measured.  For sampled parity
 * checks of large layers. */
int orc_conv2d_rows(const uint8_t* q, int32_t bits, float sx, int64_t B, int64_t H,
                    int64_t W, int64_t C, const uint8_t* codes, const float* alpha,
                    int64_t O, int32_t R, int32_t S, int32_t sh, int32_t sw,
                    int32_t ph, int32_t pw, int32_t G, const int64_t* rows,
                    int64_t nrows, int32_t nthreads, float* y, double* mag);

int orc_gemm(const uint8_t* q, int32_t bits, float sx, int64_t M, int64_t K,
             const uint8_t* codes, const float* alpha, int64_t O, int32_t G,
             int32_t nthreads, float* y);

/* Sec. 4: alpha[0..n) quantized to a `bits`-bit (8|4) signed dynamic fixed
 * point with one fractional length for the whole layer.  With amax the
 * largest alpha: integer length il = ceil(log2 amax) + 1, fl = bits - il,
 * A[i] = clamp(rint(alpha[i] * 2^fl), 0, 2^(bits-1) - 1), so the quantized
 * scale is A * 2^-fl.  amax = 0: fl = 0 and every A is 0.
 * ORC_ERR_NONFINITE for NaN, Inf or a negative alpha. */
int orc_dfp_alpha(const float* alpha, int64_t n, int32_t bits, int8_t* A,
                  int32_t* fl);

/* y[m][o] = fp32( double(S) * (double(s_x) * 2^-fl) ) with the exact
 * integer S = sum_k A[o][k/G] * t[o][k] * a[m][k]; rows as in orc_conv2d.
 * (For |S| < 2^29 the double product is exact, so y is the correctly
 * rounded value of s_x * 2^-fl * S.) */
int orc_conv2d_dfp(const uint8_t* q, int32_t bits, float sx, int64_t B,
                   int64_t H, int64_t W, int64_t C, const uint8_t* codes,
                   const int8_t* A, int32_t fl, int64_t O, int32_t R,
                   int32_t S, int32_t sh, int32_t sw, int32_t ph, int32_t pw,
                   int32_t G, int64_t row0, int64_t nrows, int32_t nthreads,
                   float* y);

int orc_gemm_dfp(const uint8_t* q, int32_t bits, float sx, int64_t M,
                 int64_t K, const uint8_t* codes, const int8_t* A, int32_t fl,
                 int64_t O, int32_t G, int32_t nthreads, float* y);

/* Sec. 4 (first layer at 8w-8a): w[0..n) quantized to a signed 8-bit
 * dynamic fixed point with one fractional length for the layer.  With wmax
 * the largest |w|: il = ceil(log2 wmax) + 1, fl = 8 - il,
 * W8[i] = clamp(rint(w[i] * 2^fl), -128, 127); wmax = 0: fl = 0, W8 = 0.
 * ORC_ERR_NONFINITE for NaN or Inf. */
int orc_w8_quantize(const float* w, int64_t n, int8_t* W8, int32_t* fl);

/* y[m][o] = fp32( double(S) * (double(s_x) * 2^-fl) ) with the exact integer
 * S = sum_{c,r,s} W8[o][c][r][s] * a[m][(r*S + s)*C + c] (W8 in the weights'
 * [O][C][R][S] order); rows as in orc_conv2d. */
int orc_conv2d_w8(const uint8_t* q, int32_t bits, float sx, int64_t B,
                  int64_t H, int64_t W, int64_t C, const int8_t* W8,
                  int32_t fl, int64_t O, int32_t R, int32_t S, int32_t sh,
                  int32_t sw, int32_t ph, int32_t pw, int64_t row0,
                  int64_t nrows, int32_t nthreads, float* y);

int orc_max_threads(void);

#ifdef __cplusplus
}
#endif
#endif
