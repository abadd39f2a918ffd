/*
 * fgq.h -- C ABI of libfgq.so: Fine-Grained Quantization (FGQ) ternary
 * inference on AMD Instinct MI355X (gfx950).
 *
 * Method: Mellempudi et al., "Ternary Neural Networks with Fine-Grained
 * Quantization" (arXiv 1705.01462).  Weights are ternarized in groups of G
 * consecutive input channels at each filter tap (Sec. 3.2, Fig. 2); every
 * group carries its own fp32 scale alpha and ternary codes t in {-1,0,+1}
 * (Sec. 3, Eq. (5)); activations are quantized to unsigned 8 or 4 bits with
 * one scale s_x per tensor (Sec. 4); a layer computes
 *
 *     y[m][o] = s_x * sum_g alpha[o][g] * P[m][o][g],
 *     P[m][o][g] = sum_{k in group g} t[o][k] * q[m][k]      (exact integer)
 *
 * (Eq. (2) applied to a convolution or fully-connected layer; one multiply
 * per group of G accumulations, Sec. 4 Discussion).
 *
 * General conventions
 *  - Every tensor pointer is a DEVICE pointer owned by the caller; the
 *    library never allocates, frees or keeps device memory of its own.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Calls enqueue work on it and return without waiting, except
 *    fgq_ternarize, which synchronizes the stream (offline preparation that
 *    must report non-finite weights).
 *  - Arguments are validated on the host before anything is enqueued; on
 *    any error nothing is launched and the outputs are untouched.
 *  - No C++ exception crosses this interface.  Calls on distinct streams
 *    with distinct buffers are thread-safe.
 *  - Shapes are int64 and must be positive unless stated otherwise.
 *
 * Layouts
 *  - Weights (input of fgq_ternarize): fp32 [O][C][R][S].
 *  - Reduction index k = (r*S + s)*C + c, K = R*S*C (a GEMM is a 1x1 conv,
 *    K = C).  Group g = k / G; G must divide C, so a group never straddles
 *    two taps.
 *  - Codes: 2 bits per weight, row o holds fgq_codes_bytes(1, K) bytes;
 *    weight k sits in bits [2(k%4), 2(k%4)+1] of byte k/4 of its row;
 *    00 = 0, 01 = +1, 11 = -1; 10 is never written.  Bits past K in the
 *    last byte of a row are zero.
 *  - alpha (and delta): fp32 [O][K/G].
 *  - Activations q: NHWC.  bits=8: one uint8 per value.  bits=4: two values
 *    per byte, element 2j in the low nibble, 2j+1 in the high nibble; C must
 *    then be even.  Real value = s_x * q, with no zero point.
 *  - Output y: fp32 NHWC [B][Ho][Wo][O] (GEMM: [M][O]),
 *    Ho = (H + 2*pad_h - R)/stride_h + 1, Wo likewise; out-of-image taps
 *    read q = 0.
 *  - s_x is a device fp32 scalar so that quantize -> conv needs no host sync.
 */
#ifndef FGQ_H
#define FGQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t fgq_status;
enum {
  FGQ_OK = 0,
  FGQ_ERR_NULL = 1,        /* a required pointer is NULL */
  FGQ_ERR_SHAPE = 2,       /* non-positive or inconsistent sizes */
  FGQ_ERR_GROUP = 3,       /* G < 1 or G does not divide C (or K) */
  FGQ_ERR_BITS = 4,        /* bits not 8|4, or odd C / n with bits=4 */
  FGQ_ERR_NONFINITE = 5,   /* fgq_ternarize met NaN or Inf weights (the
                              fixed-point calls: NaN, Inf or negative alpha;
                              the 8-bit weights: NaN or Inf) */
  FGQ_ERR_HIP = 6,         /* HIP runtime error (also: no device) */
  FGQ_ERR_UNSUPPORTED = 7, /* method or path not available for the shape */
  FGQ_ERR_WORKSPACE = 8,   /* workspace missing or too small */
  FGQ_ERR_RANGE = 9        /* fgq_prepare_weights: the group scales of some
                              output channel spread too widely for the folded
                              layout to meet its accuracy bound; run the layer
                              without a prepared buffer (direct kernel) */
};

/* Ternarization methods of fgq_ternarize. */
enum {
  FGQ_TERN_EXACT = 0,     /* Eq. (5) solved exactly by exhaustive threshold
                             search (the brute-force solve of Sec. 3.1/4) */
  FGQ_TERN_EXP_LEMMA = 1, /* Lemma 1: Delta = mean |w| of the group */
  /* 2: the asymmetric thresholds of Eq. (3)-(4), see fgq_ternarize_asym */
  FGQ_TERN_GAUSS = 3,     /* Delta = 0.612... rms(w) of the group: the
                             threshold that maximises Eq. (5) in expectation
                             for Gaussian weights (Sec. 3.1) */
  FGQ_TERN_KS = 4         /* per layer, FGQ_TERN_EXP_LEMMA or FGQ_TERN_GAUSS,
                             whichever reference law the Kolmogorov-Smirnov
                             test finds closer (Sec. 3.1; fgq_ks_distances) */
};

/* Human-readable name of a status code (static string, never NULL). */
const char* fgq_status_string(fgq_status s);

/* Interface version; bumped on any incompatible change of this header. */
int32_t fgq_abi_version(void);

/*
 * fgq_check_violations -- the bounds checks of the checking build.
 * libfgq_check.so is the same library compiled with -DFGQ_CHECK: every
 * global-memory load of the kernels that goes through a buffer descriptor
 * is tested for the one case the hardware's range check does not cover (a
 * vector offset in range carried past the end by the scalar offset), and
 * every output, split-sum and code store is tested against the extent of
 * what it writes.  A failing access is suppressed (the load reads zeros,
 * the store is skipped) and counted.  This call waits for the current
 * device, then returns in *count the number of such accesses since the
 * previous call (and in *first_site / *first_offset, when not NULL, the
 * kind of access and the byte or element offset of the first: 1
 * activations, 2 weight planes, 3 codes, 4 scale bytes, 5 group scales,
 * 6 offset terms, 7 partial maxima, 8 layer outputs, 9 split-K sums, 10
 * activation codes), and clears the counts.  For testing, not for
 * production: the normal library (libfgq.so) returns FGQ_ERR_UNSUPPORTED.
 * FGQ_ERR_NULL if count is NULL; FGQ_ERR_HIP on a runtime error.
 */
fgq_status fgq_check_violations(int64_t* count, int32_t* first_site,
                                int64_t* first_offset);

/* Number of visible HIP devices (0 when none or on runtime error). */
int32_t fgq_device_count(void);

/* Bytes of the 2-bit code array of an [O][K] weight matrix: O*ceil(K/4). */
size_t fgq_codes_bytes(int64_t O, int64_t K);

/* Number of groups O*K/G, or -1 when G does not divide K. */
int64_t fgq_group_count(int64_t O, int64_t K, int32_t G);

/*
 * fgq_ternarize -- per-group threshold Delta and scale alpha (Sec. 3, Eq. (1);
 * Sec. 3.1, Eq. (2) and Eq. (5); Lemma 1 for method 1), packed to codes.
 *
 * For each group of G weights w (G consecutive input channels at one (o,r,s),
 * Sec. 3.2): with magnitudes sorted in decreasing order (ties by channel),
 * S_j the fp64 sum of the j largest non-zero magnitudes and f_j = S_j^2 / j,
 * the kept count J is the first j maximising f_j; alpha = fp32(S_J / J),
 * Delta = the (J+1)-th largest magnitude (0 if all are kept), t = sign(w) on
 * the J largest and 0 elsewhere.  An all-zero group gets alpha = Delta = 0.
 * Method FGQ_TERN_EXP_LEMMA: Delta = fp32(mean |w|), kept iff |w| > Delta,
 * alpha = fp32(mean of the kept magnitudes) (0 if none).
 * Method FGQ_TERN_GAUSS: the same with Delta = fp32(u * sqrt(sum w^2 / G))
 * (fp64, index order), u = 0.61200318096248076, the root of
 * 2u (1 - Phi(u)) = phi(u) (for w ~ N(0, sigma) the expected objective of
 * Eq. (5) at the threshold u*sigma is proportional to phi(u)^2/(1 - Phi(u))).
 * Method FGQ_TERN_KS: FGQ_TERN_EXP_LEMMA for every group if the layer's
 * exponential K-S distance (fgq_ks_distances over all O*C*R*S weights) is
 * strictly smaller than the half-normal one, else FGQ_TERN_GAUSS.
 *
 * w      [in]  fp32 [O][C][R][S]
 * codes  [out] fgq_codes_bytes(O, R*S*C) bytes, layout above
 * alpha  [out] fp32 [O][R*S*C/G]
 * delta  [out] fp32 [O][R*S*C/G], or NULL if not wanted
 * Synchronizes `stream`.  Returns FGQ_ERR_NONFINITE if any weight is NaN or
 * Inf (outputs are then unspecified).
 */
fgq_status fgq_ternarize(const float* w, int64_t O, int64_t C, int32_t R,
                         int32_t S, int32_t G, int32_t method, uint8_t* codes,
                         float* alpha, float* delta, void* stream);

/*
 * fgq_ternarize_asym -- Eq. (3)-(4): per group, one threshold Dp for the
 * positive weights (kept iff w > Dp) and one Dn for the negative ones (kept
 * iff w < -Dn), with one scale alpha = (sum of kept |w|) / (number kept),
 * the thresholds maximising (sum of kept |w|)^2 / (number kept).  Solved
 * exhaustively: the positive and the negative magnitudes each in decreasing
 * order (ties by channel), P_a and N_b their fp64 prefix sums, every pair
 * (a, b) with a + b >= 1 scored f = (P_a + N_b)^2 / (a + b), the first
 * maximum in the order (a, then b) kept; alpha = fp32((P_a + N_b)/(a + b)),
 * Dp = the (a+1)-th positive magnitude (0 if all are kept), Dn likewise.  The
 * maximum equals that of Eq. (5) (for a given count the largest kept sum is
 * the largest magnitudes, whatever their signs), so codes match
 * FGQ_TERN_EXACT except where magnitudes tie.
 *
 * w, codes, alpha  as for fgq_ternarize
 * delta_p, delta_n [out] fp32 [O][R*S*C/G] each, or NULL if not wanted
 * Synchronizes `stream`; FGQ_ERR_NONFINITE on NaN or Inf weights.  Costs
 * (G/2)^2 steps per group on one lane: meant for groups of up to a few
 * hundred weights.
 */
fgq_status fgq_ternarize_asym(const float* w, int64_t O, int64_t C, int32_t R,
                              int32_t S, int32_t G, uint8_t* codes, float* alpha,
                              float* delta_p, float* delta_n, void* stream);

/*
 * fgq_ks_distances -- Sec. 3.1: the Kolmogorov-Smirnov distance of the weight
 * magnitudes |w| (n values, any order) to the half-normal law of N(0, sigma),
 * sigma = rms(w), CDF erf(x / (sigma sqrt 2)), and to the exponential law of
 * scale mu = mean |w| (the 1/lambda of Lemma 1), CDF 1 - exp(-x / mu), both
 * fitted by maximum likelihood.  Computed on at most 16384 magnitudes, every
 * s-th value with s = ceil(n / 16384), sorted ascending m_(1..ns):
 * sigma^2 = sum m^2 / ns, mu = sum m / ns (fp64, ascending order) and
 * D = max_i max(i/ns - F(m_(i)), F(m_(i)) - (i-1)/ns).  A sample of zeros
 * gives 0 for both.
 *
 * d [out] device fp64 [2]: D for the half-normal law, then the exponential.
 * Enqueued on `stream`.  Non-finite weights give unspecified distances.
 */
fgq_status fgq_ks_distances(const float* w, int64_t n, double* d, void* stream);

/*
 * fgq_quantize_act -- activations to unsigned `bits` (8 or 4) with one scale
 * per tensor (Sec. 4: activations quantized before each convolution).
 *
 * s = *scale_in if scale_in is not NULL (it must hold a positive finite
 * value), else s = max(max_i x_i, 0) / qmax in fp32 (s = 1 when that max is
 * 0), qmax = 255 or 15.  q_i = min(max(rint(x_i / s), 0), qmax) with IEEE
 * division and round-half-even; NaN maps to 0.  s is written to *scale_out.
 *
 * x         [in]  fp32, n values (for a conv input: NHWC, n = B*H*W*C)
 * q         [out] n bytes (bits=8) or n/2 bytes (bits=4, n even)
 * scale_out [out] device fp32 scalar
 * ws        [tmp] device workspace of fgq_quantize_ws_bytes(n) bytes, needed
 *                 only when scale_in is NULL (dynamic scale); not kept.
 */
size_t fgq_quantize_ws_bytes(int64_t n);
fgq_status fgq_quantize_act(const float* x, int64_t n, int32_t bits,
                            const float* scale_in, uint8_t* q,
                            float* scale_out, void* ws, size_t ws_bytes,
                            void* stream);

/*
 * fgq_quantize_act_noalloc -- fgq_quantize_act without a workspace, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops that must not call hipMalloc, harnesses that forbid it).
 * Same arguments and results as fgq_quantize_act (bit for bit).  The dynamic
 * scale's partial maxima go to a 4 KB array of the library's own in device
 * memory, one per device, held until the process ends (its address is looked
 * up on the first call on each device).  The maximum is 1024 partial maxima,
 * which covers every n (pass 1 runs at most 1024 blocks);
 * FGQ_ERR_WORKSPACE would report a larger need.  Nothing is allocated and
 * nothing needs to start at zero (each call writes every partial it reads).
 * Calls that overlap on one device (on different streams, or from several
 * threads) share that array and race: serialize them.
 */
fgq_status fgq_quantize_act_noalloc(const float* x, int64_t n, int32_t bits,
                                    const float* scale_in, uint8_t* q,
                                    float* scale_out, void* stream);

/*
 * fgq_prepare_weights -- per-layer constants for the matrix-core kernels
 * (built once per layer, like the ternarization itself).  The layout
 * depends on G alone:
 *
 * G = 64 with K/64 <= 160 (per-group kernel, Sec. 4: 32-bit group sums,
 * then one multiplication by the group scale per group): the 2-bit codes in
 * the kernel's operand order (expanded to int8 in registers) and alpha
 * transposed per group; 0.25 bytes per weight plus 4 bytes per group.
 *
 * Any other G (folded-scale kernel): the group scales are brought to one
 * grid per output channel: A[o][g] = rint(alpha[o][g] / h_o), with h_o the
 * smallest fp32 step keeping every A of the channel within
 * 127*(1 + 255 + 255^2), written as three balanced base-255 digits in
 * [-127, 127].  The folded weights t*digit are int8, so the layer runs as
 * three exact int8 products whose integer sums are combined exactly (for
 * G = 4 and G = 64 the convolution reads the 2-bit codes and each group's
 * three digits, 0.25 + 3/G bytes per weight, and expands them in
 * registers; for other G it reads the int8 planes); only
 * the rounding of alpha to the grid (at most h_o / 2, about 6e-8 times the
 * channel's largest alpha) and the fp32 conversions and fused multiply-adds
 * of the final combination differ from the exact formula.  3 bytes per
 * weight.
 *
 * Accuracy guard (folded layout only): the result is within 1e-5 of
 * s_x * sum_g alpha_g |P_g| for every input when each non-zero scale of a
 * channel lies within a relative 9.2e-6 of its grid value A * h_o (the
 * fp32 combination adds less than 7.75e-7 of that magnitude).  That fails only
 * for channels whose scales spread over a wide range (the grid step follows
 * the channel's largest alpha; smaller scales keep fewer bits).  The check
 * is exact, per channel, on the device; then the call returns
 * FGQ_ERR_RANGE, and the layer must run without the prepared buffer (the
 * direct kernel, exact).  The buffer is still written, with a NaN scale for
 * each failing channel, so that a layer run with it anyway gives NaN fp32
 * outputs in those channels.  A negative or non-finite alpha fails its
 * channel too.
 *
 * codes, alpha  [in]  as produced by fgq_ternarize for an [O][K] layer
 * prepared      [out] device buffer of fgq_prepared_bytes(O, K, G) bytes,
 *                     256-byte aligned; opaque; read by fgq_conv2d/fgq_gemm
 *                     with the same O, K, G.
 * Synchronizes `stream` (the folded layout's guard is read back).
 */
size_t fgq_prepared_bytes(int64_t O, int64_t K, int32_t G);
fgq_status fgq_prepare_weights(const uint8_t* codes, const float* alpha,
                               int64_t O, int64_t K, int32_t G, void* prepared,
                               size_t prepared_bytes, void* stream);

/*
 * fgq_conv2d -- FGQ convolution as an implicit GEMM (Sec. 3.2 grouping;
 * Sec. 4 low-precision pipeline with 32-bit integer accumulation):
 * y[b][ho][wo][o] = s_x * sum_g alpha[o][g] * P_g with the group sums P_g
 * taken over the input window of output pixel (b, ho, wo).
 *
 * q        [in]  activations NHWC [B][H][W][C], bits 8 or 4 (layout above)
 * sx       [in]  device fp32 scalar s_x (e.g. fgq_quantize_act's scale_out)
 * codes    [in]  2-bit codes of the [O][R][S][C] weights
 * alpha    [in]  fp32 [O][K/G]
 * prepared [in]  NULL, or the output of fgq_prepare_weights for these
 *                codes/alpha/O/K/G.  NULL selects the direct per-group
 *                kernel: exact int32 group sums (packed 4-way dot products)
 *                and an fp64 alpha epilogue, bit-identical to evaluating the
 *                formula in fp64 in group order and rounding once to fp32.
 *                Non-NULL selects a matrix-core kernel when C is a multiple
 *                of 16, q is 16-byte (bits 8) or 8-byte (bits 4) aligned and
 *                every buffer is below 2^31 bytes: the per-group kernel for
 *                G = 64 (int32 group sums, fp32 alpha epilogue, at most
 *                K/64 + 1 fp32 roundings relative to s_x*sum_g alpha_g|P_g|)
 *                and the folded-scale kernel for other G (K <= 65536);
 *                otherwise the direct kernel runs.
 * y        [out] fp32 [B][Ho][Wo][O]
 */
fgq_status fgq_conv2d(const uint8_t* q, int32_t bits, const float* sx,
                      int64_t B, int64_t H, int64_t W, int64_t C,
                      const uint8_t* codes, const float* alpha,
                      const void* prepared, int64_t O, int32_t R, int32_t S,
                      int32_t stride_h, int32_t stride_w, int32_t pad_h,
                      int32_t pad_w, int32_t G, float* y, void* stream);

/*
 * fgq_gemm -- FGQ fully-connected layer, y[m][o] = s_x * sum_g alpha[o][g] *
 * sum_{k in g} t[o][k] q[m][k]; identical to fgq_conv2d with B=1, H=M, W=1,
 * C=K, R=S=1.  q is [M][K] (bits=4: K even); y is [M][O].
 */
fgq_status fgq_gemm(const uint8_t* q, int32_t bits, const float* sx,
                    int64_t M, int64_t K, const uint8_t* codes,
                    const float* alpha, const void* prepared, int64_t O,
                    int32_t G, float* y, void* stream);

/*
 * fgq_conv2d_q / fgq_gemm_q -- the same layers with the next layer's
 * activation quantization fused into the epilogue (Sec. 4: activations are
 * quantized before each convolution; the quantization's clamp at 0 is the
 * ReLU between layers).  Instead of y, writes
 *   q_out = fgq_quantize_act(y, out_bits, scale_in = out_scale)
 * for the y that fgq_conv2d / fgq_gemm computes with the same arguments,
 * bit for bit (same kernels, same arithmetic; the quantization follows
 * fgq_quantize_act exactly).  The scale is given (a per-layer calibrated
 * scale); a dynamic scale needs the whole output first and is not fused.
 *
 * out_bits  [in]  8 or 4 (4 needs O even)
 * out_scale [in]  device fp32 scalar, a positive finite value
 * q_out     [out] NHWC [B][Ho][Wo][O] bytes (8) or [B][Ho][Wo][O/2] (4: the
 *                 even channel in the low nibble) -- the next layer's q
 */
fgq_status fgq_conv2d_q(const uint8_t* q, int32_t bits, const float* sx,
                        int64_t B, int64_t H, int64_t W, int64_t C,
                        const uint8_t* codes, const float* alpha,
                        const void* prepared, int64_t O, int32_t R, int32_t S,
                        int32_t stride_h, int32_t stride_w, int32_t pad_h,
                        int32_t pad_w, int32_t G, int32_t out_bits,
                        const float* out_scale, uint8_t* q_out, void* stream);
fgq_status fgq_gemm_q(const uint8_t* q, int32_t bits, const float* sx,
                      int64_t M, int64_t K, const uint8_t* codes,
                      const float* alpha, const void* prepared, int64_t O,
                      int32_t G, int32_t out_bits, const float* out_scale,
                      uint8_t* q_out, void* stream);

/*
 * fgq_conv2d_residual -- the convolution with a residual block's shortcut
 * addition and ReLU fused into its epilogue (the residual networks of the
 * Sec. 4 experiments end each block with such an addition; it is not part of
 * the FGQ layer itself).  Writes
 *   y = max(yc + res, 0)   elementwise, the fp32 sum rounded once,
 * where yc is the fp32 output fgq_conv2d computes with the same arguments
 * (same kernels, same arithmetic; a NaN sum stays NaN), so the result equals
 * fgq_conv2d followed by an fp32 addition and a ReLU, bit for bit, without
 * the separate passes over the output.
 *
 * res [in]  fp32 [B][Ho][Wo][O] device tensor, the shortcut (the block input
 *           or its projection); may be y itself (in place), must not
 *           partially overlap it
 * y   [out] fp32 [B][Ho][Wo][O]
 * Other arguments and errors as fgq_conv2d; FGQ_ERR_NULL if res is NULL.
 */
fgq_status fgq_conv2d_residual(const uint8_t* q, int32_t bits, const float* sx,
                               int64_t B, int64_t H, int64_t W, int64_t C,
                               const uint8_t* codes, const float* alpha,
                               const void* prepared, int64_t O, int32_t R,
                               int32_t S, int32_t stride_h, int32_t stride_w,
                               int32_t pad_h, int32_t pad_w, int32_t G,
                               const float* res, float* y, void* stream);

/*
 * fgq_conv2d_residual_q -- fgq_conv2d_residual that also writes the codes of
 * its output, the next block's input (Sec. 4: activations are quantized
 * before each convolution), at a given scale:
 *   y     = max(yc + res, 0)                             as fgq_conv2d_residual
 *   q_out = fgq_quantize_act(y, out_bits, scale_in = out_scale)
 * both bit for bit, from one epilogue.  Arguments as fgq_conv2d_residual,
 * plus out_bits / out_scale / q_out as fgq_conv2d_q (out_bits 4 needs O even).
 */
fgq_status fgq_conv2d_residual_q(const uint8_t* q, int32_t bits, const float* sx,
                                 int64_t B, int64_t H, int64_t W, int64_t C,
                                 const uint8_t* codes, const float* alpha,
                                 const void* prepared, int64_t O, int32_t R,
                                 int32_t S, int32_t stride_h, int32_t stride_w,
                                 int32_t pad_h, int32_t pad_w, int32_t G,
                                 const float* res, float* y, int32_t out_bits,
                                 const float* out_scale, uint8_t* q_out,
                                 void* stream);

/*
 * Fixed-point group scales (Sec. 4: the scaling factors are quantized to an
 * 8- or 4-bit fixed point; 32-bit accumulation).
 *
 * fgq_dfp_alpha -- alpha quantized to a `bits`-bit (8|4) signed dynamic
 * fixed point with one fractional length for the whole layer: with amax the
 * largest alpha, integer length il = ceil(log2 amax) + 1, fl = bits - il,
 * A = clamp(rint(alpha * 2^fl), 0, 2^(bits-1) - 1) (ties to even), so the
 * quantized scale is A * 2^-fl; amax = 0 gives fl = 0 and A = 0.
 *   alpha [in]  fp32, n values (e.g. a layer's [O][K/G] scales)
 *   A     [out] int8, n values
 *   fl    [out] device int32 scalar
 * Synchronizes `stream`; FGQ_ERR_NONFINITE if an alpha is NaN, Inf or
 * negative (outputs then unspecified).
 *
 * fgq_prepare_weights_dfp -- the constants of the layer with those scales:
 * the int8 weights A[o][g(k)] * t[o][k] (one plane, the folded kernel's
 * operand order), their uint8 offset term, fl, the dequantized scales and
 * the codes A.  1 byte per weight plus 5 per group.  prepared: device buffer of
 * fgq_prepared_bytes_dfp(O, K, G) bytes, 256-byte aligned, opaque.
 * Synchronizes `stream`; FGQ_ERR_NONFINITE as for fgq_dfp_alpha.
 *
 * fgq_conv2d_dfp / fgq_gemm_dfp -- the layer
 *   y = fp32( double(S) * (double(s_x) * 2^-fl) ),
 *   S[m][o] = sum_k A[o][g(k)] t[o][k] q[m][k]   (exact int32),
 * which is the correctly rounded value of s_x 2^-fl S whenever |S| < 2^29
 * (K < 16577 for uint8).  Bit-identical on every path: the one-plane
 * matrix-core kernel when C % 16 == 0 (or C = 4, 8), q is aligned as for
 * fgq_conv2d and K <= 65536; otherwise the direct kernel on the dequantized
 * scales.  Arguments as for fgq_conv2d / fgq_gemm, with the scales taken
 * from `prepared` (codes are still read by the direct path).
 *   out_bits  [in]  0: out is fp32 y; 8 or 4: out receives the codes of
 *                   fgq_quantize_act(y, out_bits, scale_in = out_scale),
 *                   laid out as q_out of fgq_conv2d_q (4 needs O even)
 *   out_scale [in]  device fp32 scalar when out_bits != 0, else ignored
 */
fgq_status fgq_dfp_alpha(const float* alpha, int64_t n, int32_t bits,
                         int8_t* A, int32_t* fl, void* stream);
size_t fgq_prepared_bytes_dfp(int64_t O, int64_t K, int32_t G);
fgq_status fgq_prepare_weights_dfp(const uint8_t* codes, const float* alpha,
                                   int64_t O, int64_t K, int32_t G,
                                   int32_t alpha_bits, void* prepared,
                                   size_t prepared_bytes, void* stream);
fgq_status fgq_conv2d_dfp(const uint8_t* q, int32_t bits, const float* sx,
                          int64_t B, int64_t H, int64_t W, int64_t C,
                          const uint8_t* codes, const void* prepared,
                          int64_t O, int32_t R, int32_t S, int32_t stride_h,
                          int32_t stride_w, int32_t pad_h, int32_t pad_w,
                          int32_t G, int32_t out_bits, const float* out_scale,
                          void* out, void* stream);
fgq_status fgq_gemm_dfp(const uint8_t* q, int32_t bits, const float* sx,
                        int64_t M, int64_t K, const uint8_t* codes,
                        const void* prepared, int64_t O, int32_t G,
                        int32_t out_bits, const float* out_scale, void* out,
                        void* stream);

/*
 * fgq_conv2d_dfp_residual -- fgq_conv2d_dfp with a residual block's shortcut
 * addition and ReLU in its epilogue, as fgq_conv2d_residual does for
 * fgq_conv2d: y = max(yd + res, 0) for the fp32 output yd of fgq_conv2d_dfp
 * (the sum rounded once), bit for bit.  out_bits 0: y only; 8 or 4: also
 * q_out = fgq_quantize_act(y, out_bits, scale_in = out_scale) (4 needs O
 * even), the next block's input.  res: fp32 [B][Ho][Wo][O], may be y
 * itself, must not partially overlap it.  Other arguments as
 * fgq_conv2d_dfp; out_scale and q_out are ignored when out_bits is 0.
 */
fgq_status fgq_conv2d_dfp_residual(const uint8_t* q, int32_t bits, const float* sx,
                                   int64_t B, int64_t H, int64_t W, int64_t C,
                                   const uint8_t* codes, const void* prepared,
                                   int64_t O, int32_t R, int32_t S,
                                   int32_t stride_h, int32_t stride_w,
                                   int32_t pad_h, int32_t pad_w, int32_t G,
                                   const float* res, float* y, int32_t out_bits,
                                   const float* out_scale, uint8_t* q_out,
                                   void* stream);

/*
 * GEMMs with split K, for fully-connected layers at small batch (few rows,
 * long K: the rows and channels alone would occupy few compute units).
 *
 * fgq_gemm_ws / fgq_gemm_dfp_ws -- the same results as fgq_gemm (or
 * fgq_gemm_q, by out_bits) and fgq_gemm_dfp, bit for bit: when the
 * matrix-core kernel runs (prepared given, shape as for fgq_gemm, and for
 * fgq_gemm_ws the folded layout, i.e. G != 64 or K/64 > 160), the K steps
 * are divided among workgroups that write their int32 sums to `ws`, and a
 * second kernel adds them in a fixed order and applies the usual epilogue.
 * With M <= 64, K % 16 == 0 and G in {4, 8, 16, 32, 64, 128} (and, for
 * fgq_gemm_ws, the folded layout) the kernel reads the weights as the 2-bit
 * codes plus, per group, the scale code A (fgq_gemm_dfp_ws) or the three
 * digits of the scale (fgq_gemm_ws), all stored by the prepare call in the
 * kernel's operand order, and expands them to int8 weights in registers;
 * such shapes always use the workspace.
 *   out_bits / out_scale / out  as for fgq_conv2d_dfp
 *   ws        [tmp] device buffer of fgq_gemm_ws_bytes(M, K, O, G,
 *                   fixed_point) bytes (4-byte aligned, 16-byte aligned
 *                   for the fastest stores; fixed_point = 1 for
 *                   fgq_gemm_dfp_ws), not kept between calls; may be NULL
 *                   when that size is 0 (K is then not split).
 * FGQ_ERR_WORKSPACE if a needed workspace is missing or too small.  The
 * split depends on the device's compute-unit count: query the size on the
 * device that runs the call.
 */
size_t fgq_gemm_ws_bytes(int64_t M, int64_t K, int64_t O, int32_t G,
                         int32_t fixed_point);
fgq_status fgq_gemm_ws(const uint8_t* q, int32_t bits, const float* sx,
                       int64_t M, int64_t K, const uint8_t* codes,
                       const float* alpha, const void* prepared, int64_t O,
                       int32_t G, int32_t out_bits, const float* out_scale,
                       void* out, void* ws, size_t ws_bytes, void* stream);
fgq_status fgq_gemm_dfp_ws(const uint8_t* q, int32_t bits, const float* sx,
                           int64_t M, int64_t K, const uint8_t* codes,
                           const void* prepared, int64_t O, int32_t G,
                           int32_t out_bits, const float* out_scale,
                           void* out, void* ws, size_t ws_bytes,
                           void* stream);

/*
 * First layer at 8-bit weights (Sec. 4 keeps the first layer at 8w-8a).
 *
 * fgq_prepare_weights_w8 -- the weights w (fp32 [O][C][R][S]) as a signed
 * 8-bit dynamic fixed point with one fractional length for the layer: with
 * wmax = max |w|, fl = 8 - (ceil(log2 wmax) + 1), W8 = clamp(rint(w * 2^fl),
 * -128, 127) (ties to even; wmax = 0 gives fl = 0), stored in the layout of
 * fgq_prepare_weights_dfp.  prepared: fgq_prepared_bytes_w8(O, C, R, S)
 * bytes, 256-byte aligned.  Synchronizes `stream`; FGQ_ERR_NONFINITE if a
 * weight is NaN or Inf.
 *
 * fgq_conv2d_w8 -- y = fp32( double(S) * (double(s_x) * 2^-fl) ),
 * S[m][o] = sum_k W8[o][k] q[m][k] (exact int32), on the one-plane
 * matrix-core kernel; needs C % 16 == 0 or C = 4, 8 (a first layer with
 * its 3 image channels padded to 4), q aligned as for fgq_conv2d and
 * R*S*C <= 65536, else FGQ_ERR_UNSUPPORTED.  out_bits / out_scale / out as
 * for fgq_conv2d_dfp.
 */
size_t fgq_prepared_bytes_w8(int64_t O, int64_t C, int32_t R, int32_t S);
fgq_status fgq_prepare_weights_w8(const float* w, int64_t O, int64_t C,
                                  int32_t R, int32_t S, void* prepared,
                                  size_t prepared_bytes, void* stream);
fgq_status fgq_conv2d_w8(const uint8_t* q, int32_t bits, const float* sx,
                         int64_t B, int64_t H, int64_t W, int64_t C,
                         const void* prepared, int64_t O, int32_t R, int32_t S,
                         int32_t stride_h, int32_t stride_w, int32_t pad_h,
                         int32_t pad_w, int32_t out_bits,
                         const float* out_scale, void* out, void* stream);

/*
 * fgq_group_sums -- the exact integer group sums P[m][o][g] (Sec. 4: 32-bit
 * accumulation) of fgq_conv2d's geometry for output rows m in
 * [row0, row0 + nrows), m = (b*Ho + ho)*Wo + wo.
 *
 * P [out] int32 [nrows][O][K/G]
 */
fgq_status fgq_group_sums(const uint8_t* q, int32_t bits, int64_t B,
                          int64_t H, int64_t W, int64_t C,
                          const uint8_t* codes, int64_t O, int32_t R,
                          int32_t S, int32_t stride_h, int32_t stride_w,
                          int32_t pad_h, int32_t pad_w, int32_t G,
                          int64_t row0, int64_t nrows, int32_t* P,
                          void* stream);

/*
 * Measurement utility (not part of the method): the rate of the int8 matrix
 * instruction the layer kernels use, for reporting kernels against a
 * measured peak next to the published one.
 *
 * fgq_probe_mfma_i8 -- launches `blocks` workgroups of 256 threads; each
 * wave issues `iters` rounds of four independent 32x32x32 int8 matrix
 * instructions (2 * 32768 int8 operations each), i.e. blocks * iters *
 * 16 * 65536 operations in all, then writes one int32 per thread to `out`
 * (a sink that keeps the work alive; values meaningless).  out must hold
 * blocks * 256 int32 (out_elems); FGQ_ERR_SHAPE for blocks or iters < 1 or
 * a smaller out.  Enqueued on `stream`.
 */
fgq_status fgq_probe_mfma_i8(int32_t blocks, int32_t iters, int32_t* out,
                             int64_t out_elems, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* FGQ_H */
