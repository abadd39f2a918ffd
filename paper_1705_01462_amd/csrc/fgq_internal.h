// fgq_internal.h -- internal declarations shared by the libfgq sources.
// Not installed; the public interface is include/fgq.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "bufcheck.h"
#include "fgq.h"

#define FGQ_TRY_HIP(expr)                      \
  do {                                         \
    hipError_t fgq_e_ = (expr);                \
    if (fgq_e_ != hipSuccess) return FGQ_ERR_HIP; \
  } while (0)

namespace fgq {

// Geometry of an implicit-GEMM convolution (a GEMM is B=1, H=M, W=1, R=S=1).
struct ConvGeom {
  int64_t B, H, W, C, O, Ho, Wo, M, K;
  int32_t R, S, sh, sw, ph, pw, G, bits;
};

// Where a layer's result goes: fp32 y (bits = 0), or the layer's output
// fused with the next layer's activation quantization: unsigned `bits` codes
// of every output value with the device scale *scale, NHWC like y (bits 4:
// two channels per byte, the even channel in the low nibble; O even); or
// (bits = 2) fp32 y = max(layer + res, 0) with res an fp32 tensor of y's
// shape, a residual block's shortcut addition and ReLU; or (bits = 2 | 8,
// 2 | 4) that y and also its codes in q.
struct LayerOut {
  float* y;
  uint8_t* q;
  const float* scale;
  int32_t bits;
  const float* res = nullptr;
};

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

inline fgq_status last_launch() {
  return hipGetLastError() == hipSuccess ? FGQ_OK : FGQ_ERR_HIP;
}

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// Layout of the buffer written by fgq_prepare_weights (offsets in bytes).
// Two kinds, chosen by G alone:
//  * group (G = 64 and at most kGroupMaxGroups groups per channel): the
//    per-group kernel.
//      planes : the 2-bit codes in the kernel's operand order
//               [O32/32][Kp/128][64 lanes][4 words of 16 codes] (prepare.hip)
//      alpha  : fp32 [Kp/64][O32], alpha of group k/64 of channel o
//  * fold (every other G): the folded-scale kernel.
//      planes : int8 folded digits t*d_j (j = 0 least significant),
//               [O32/32][Kp/64][3 planes][2 K halves][64 lanes][16 bytes]
//      bias   : int32 [3][O]  128 * sum_k plane_j[o][k] (uint8 offset term)
//      scale  : fp32  [O]     the grid step h_o (NaN: the channel fails the accuracy guard)
//      xcodes, xacodes (G a power of two in 4..128): the 2-bit codes and the
//               three digits of each group's scale in the codes-expanding
//               order (xlayout.h; digits plane-major), read by the GEMM at
//               small batch and, for G = 4 and 64, by the convolution
// A third kind is written by fgq_prepare_weights_dfp (any G), for the layer
// with fixed-point group scales:
//      header : int32 fl, the fractional length of the layer's scales
//      planes : int8 A[o][g(k)] * t[o][k], one plane,
//               [O32/32][Kp/64][1 plane][2 K halves][64 lanes][16 bytes]
//      bias   : int32 [O]     128 * sum_k plane[o][k]
//      alpha  : fp32 [O][K/G] the dequantized scales A * 2^-fl (direct path)
//      xcodes, xacodes (G a power of two in 4..128): the 2-bit codes and the
//               scale codes A in the order of the GEMM that expands them in
//               registers (dfpx.hip; layout there)
// In the fragment order, lane l of (channel tile, 64-wide K block, plane,
// half) holds channel 32*tile + l%32, k = 64*block + 32*half + 16*(l/32) +
// [0, 16), so each wave-wide 16-byte load is one contiguous kilobyte.
// Channels >= O, k >= K (and their alpha) are zero; Kp is a multiple of 128.
enum PrepKind { kPrepFold = 0, kPrepGroup = 1, kPrepDfp = 2 };
struct PreparedLayout {
  int kind;
  int64_t O32, Kp, nks, planes_off, bias_off, scale_off, alpha_off, xcodes_off, xacodes_off, total;
};
constexpr int64_t kFoldKStep = 64;
constexpr int64_t kFoldTileBytes = 3 * 2 * 64 * 16;  // one channel tile, one K block
constexpr int64_t kDfpHeaderBytes = 256;
// Largest K of the int8 folded kernels: with uint8 activations the int32
// accumulator holds up to 255 * 127 * K, below 2^31 for K <= 65536.
constexpr int64_t kFoldMaxK = 65536;
// The per-group kernel accumulates one fp32 product per group; with at most
// 160 groups its rounding error stays below 1e-5 of the summand magnitude.
constexpr int64_t kGroupMaxGroups = 160;
// Accuracy guard of the folded layout.  With every group scale on the
// channel's grid, Ahat_g = A_g h (A_g = rint(alpha_g / h)), the integer sums
// are exact and S_j = sum_g d_j(g) P_g, so the fp32 combination of the three
// digit sums (three conversions, c0 = s_x h and two coefficients c0 255^j
// rounded, a product and two fused multiply-adds) is within 13 * 2^-24 <
// kFoldCombineRel of s_x * sum_g Ahat_g |P_g| (balanced digits have
// sum_j 255^j |d_j| < 3 A).  A channel whose scales all satisfy
// |Ahat_g - alpha_g| <= kFoldMaxRel * alpha_g therefore meets 1e-5 of
// s_x * sum_g alpha_g |P_g| for every input:
// 9.2e-6 + 7.75e-7 * (1 + 9.2e-6) < 1e-5.
constexpr double kFoldMaxRel = 9.2e-6;
constexpr double kFoldCombineRel = 7.75e-7;
PreparedLayout prepared_layout(int64_t O, int64_t K, int32_t G);
PreparedLayout prepared_layout_dfp(int64_t O, int64_t K, int32_t G);

// Launchers (return FGQ_OK or FGQ_ERR_HIP); arguments already validated.
fgq_status launch_ternarize(const float* w, int64_t O, int64_t C, int32_t R, int32_t S, int32_t G,
                            int32_t method, uint8_t* codes, float* alpha, float* delta, float* delta_n,
                            hipStream_t st);
// Eq. (3)-(4) as a ternarize method (fgq_ternarize_asym; delta = Dp,
// delta_n = Dn).
constexpr int32_t kTernAsym = 2;
// K-S distances (d, nullable device [2]) and the rule they pick (pick,
// nullable device int32), ternarize.hip; the sample size.
constexpr int kKsSample = 16384;
fgq_status launch_ks(const float* w, int64_t n, double* d, int32_t* pick, hipStream_t st);
fgq_status launch_quantize(const float* x, int64_t n, int32_t bits,
                           const float* scale_in, uint8_t* q, float* scale_out,
                           float* partials, int32_t npart, hipStream_t st);
int32_t quantize_partials(int64_t n);
// The allocation-free quantization (fgq_quantize_act_noalloc) keeps pass 1's
// partial maxima in a file-scope device array of kQuantScratchFloats floats
// (4 KB per device, held until the process ends); quantize_scratch gives its
// address on the current device.
constexpr int32_t kQuantScratchFloats = 1024;
constexpr int kMaxDevices = 64;
fgq_status quantize_scratch(float** out);
fgq_status launch_exact_conv(const uint8_t* q, const float* sx,
                             const uint8_t* codes, const float* alpha,
                             const ConvGeom& g, const LayerOut& out, hipStream_t st);
fgq_status launch_group_sums(const uint8_t* q, const uint8_t* codes,
                             const ConvGeom& g, int64_t row0, int64_t nrows,
                             int32_t* P, hipStream_t st);
fgq_status launch_prepare(const uint8_t* codes, const float* alpha, int64_t O,
                          int64_t K, int32_t G, void* prepared,
                          hipStream_t st);
// Fixed-point group scales: the layer exponent into *fl (INT32_MIN when an
// alpha is NaN, Inf or negative) and the codes A (A may be NULL).
fgq_status launch_dfp_alpha(const float* alpha, int64_t n, int32_t bits, int8_t* A,
                            int32_t* fl, hipStream_t st);
// First layer at 8-bit weights: the fixed-point prepared layout (with one
// group per tap, G = C) with W8 as the plane.
fgq_status launch_prepare_w8(const float* w, int64_t O, int64_t C, int32_t R, int32_t S,
                             void* prepared, hipStream_t st);
fgq_status launch_prepare_dfp(const uint8_t* codes, const float* alpha, int64_t O,
                              int64_t K, int32_t G, int32_t alpha_bits, void* prepared,
                              hipStream_t st);
// Folded-scale int8 MFMA kernel (prepared layout of kind fold); callers
// check fold_supported first.  The dfp variant runs the one-plane layer of
// kind dfp on the same kernel.
bool fold_supported(const ConvGeom& g, const uint8_t* q);
fgq_status launch_fold_conv(const uint8_t* q, const float* sx,
                            const void* prepared, const ConvGeom& g, const LayerOut& out,
                            hipStream_t st);
bool fold_dfp_supported(const ConvGeom& g, const uint8_t* q);
fgq_status launch_fold_dfp_conv(const uint8_t* q, const float* sx,
                                const void* prepared, const ConvGeom& g, const LayerOut& out,
                                hipStream_t st);
// Split K for the folded kernels (splitk.hip): the number of splits for an
// M x K x O product (1: none) and its steps per split; the split launches
// write int32 sums to ws [splits][planes][M][O] and reduce them into `out`.
int32_t splitk_splits(int64_t M, int64_t K, int64_t O, int32_t* steps_per_split);
fgq_status launch_fold_splitk(const uint8_t* q, const float* sx, const void* prepared, const ConvGeom& g,
                              const LayerOut& out, int32_t splits, int32_t steps_per_split, int32_t* ws,
                              hipStream_t st);
fgq_status launch_fold_dfp_splitk(const uint8_t* q, const float* sx, const void* prepared, const ConvGeom& g,
                                  const LayerOut& out, int32_t splits, int32_t steps_per_split, int32_t* ws,
                                  hipStream_t st);
// The fixed-point GEMM at few rows (M <= kDfpxMaxM), weights expanded from
// the 2-bit codes and the scale codes in registers (dfpx.hip): its own K
// split (dfpx_splits), int32 sums in ws [splits][M][O], the same reduction.
constexpr int64_t kDfpxMaxM = 64;
// Scale-code bytes per lane and 128-wide K step in that order (0: no such
// regions for this G).
inline int64_t dfpx_acode_bytes(int32_t G) {
  return (G == 4 || G == 8 || G == 16 || G == 32 || G == 64) ? 64 / G : (G == 128 ? 1 : 0);
}
bool dfpx_shape_ok(int64_t M, int64_t K, int64_t O, int32_t G);
bool dfpx_supported(const ConvGeom& g, const uint8_t* q);
int32_t dfpx_splits(int64_t M, int64_t K, int64_t O, int32_t G, int32_t* steps_per_split);
fgq_status launch_dfpx_splitk(const uint8_t* q, const float* sx, const void* prepared,
                              const ConvGeom& g, const LayerOut& out, int32_t* ws, hipStream_t st);
// The same kernel on the folded layout (fp32 scales as three int8 digit
// planes), int32 sums in ws [splits][3][M][O], the folded reduction.
fgq_status launch_foldx_splitk(const uint8_t* q, const float* sx, const void* prepared,
                               const ConvGeom& g, const LayerOut& out, int32_t* ws, hipStream_t st);
fgq_status launch_splitk_reduce(const int32_t* part, int32_t splits, bool dfp, int64_t M, int64_t O,
                                const float* sx, const float* scale, const int32_t* fl, const LayerOut& out,
                                hipStream_t st);
// Per-group int8 MFMA kernel with an fp32 alpha epilogue (G = 64).
bool group_supported(const ConvGeom& g, const uint8_t* q);
fgq_status launch_group_conv(const uint8_t* q, const float* sx,
                             const void* prepared, const ConvGeom& g, const LayerOut& out,
                             hipStream_t st);

}  // namespace fgq
