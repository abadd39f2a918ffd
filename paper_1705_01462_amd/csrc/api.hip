// api.hip -- the extern "C" boundary of libfgq.so (declared in include/fgq.h):
// host-side validation, then kernel selection and launch on the caller's
// stream.  No allocation, no hidden device state.
#include <stdlib.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "fgq_internal.h"

using namespace fgq;

#ifdef FGQ_CHECK
namespace fgq {
namespace {
std::mutex& check_mutex() {
  static std::mutex m;
  return m;
}
std::vector<const void*>& check_records() {
  static std::vector<const void*> v;
  return v;
}
}  // namespace

// Called at load time by every compilation unit of a checking build (no
// HIP call here: the records are looked up when they are read).
void check_register(const void* symbol) {
  std::lock_guard<std::mutex> g(check_mutex());
  check_records().push_back(symbol);
}
}  // namespace fgq
#endif

namespace {

bool conv_geom(int64_t B, int64_t H, int64_t W, int64_t C, int64_t O, int32_t R, int32_t S,
               int32_t sh, int32_t sw, int32_t ph, int32_t pw, int32_t G, int32_t bits,
               ConvGeom* g, fgq_status* err) {
  *err = FGQ_OK;
  if (bits != 8 && bits != 4) {
    *err = FGQ_ERR_BITS;
    return false;
  }
  if (B < 1 || H < 1 || W < 1 || C < 1 || O < 1 || R < 1 || S < 1 || sh < 1 || sw < 1 ||
      ph < 0 || pw < 0 || H + 2LL * ph < R || W + 2LL * pw < S) {
    *err = FGQ_ERR_SHAPE;
    return false;
  }
  if (G < 1 || C % G != 0) {
    *err = FGQ_ERR_GROUP;
    return false;
  }
  if (bits == 4 && C % 2 != 0) {
    *err = FGQ_ERR_BITS;
    return false;
  }
  g->B = B; g->H = H; g->W = W; g->C = C; g->O = O;
  g->R = R; g->S = S; g->sh = sh; g->sw = sw; g->ph = ph; g->pw = pw;
  g->G = G; g->bits = bits;
  g->Ho = (H + 2LL * ph - R) / sh + 1;
  g->Wo = (W + 2LL * pw - S) / sw + 1;
  g->M = B * g->Ho * g->Wo;
  g->K = static_cast<int64_t>(R) * S * C;
  if (g->M > (1LL << 40) || g->K > (1LL << 31) || O > (1LL << 31)) {
    *err = FGQ_ERR_SHAPE;
    return false;
  }
  return true;
}

fgq_status run_layer(const uint8_t* q, const float* sx, const uint8_t* codes,
                     const float* alpha, const void* prepared, const ConvGeom& g,
                     const LayerOut& y, void* stream) {
  hipStream_t st = as_stream(stream);
  if (prepared) {
    if (prepared_layout(g.O, g.K, g.G).kind == kPrepGroup) {
      if (group_supported(g, q)) return launch_group_conv(q, sx, prepared, g, y, st);
    } else if (fold_supported(g, q)) {
      return launch_fold_conv(q, sx, prepared, g, y, st);
    }
  }
  return launch_exact_conv(q, sx, codes, alpha, g, y, st);
}

// The layer with fixed-point scales: the one-plane folded kernel when the
// shape allows it, else the direct kernel on the dequantized scales stored
// in the prepared buffer (every alpha*P product and their fp64 sum are then
// exact, so both give fp32(double(S) * (double(s_x) * 2^-fl))).
fgq_status run_layer_dfp(const uint8_t* q, const float* sx, const uint8_t* codes,
                         const void* prepared, const ConvGeom& g, const LayerOut& y, void* stream) {
  hipStream_t st = as_stream(stream);
  if (fold_dfp_supported(g, q)) return launch_fold_dfp_conv(q, sx, prepared, g, y, st);
  const PreparedLayout L = prepared_layout_dfp(g.O, g.K, g.G);
  const float* alpha_q = reinterpret_cast<const float*>(static_cast<const char*>(prepared) + L.alpha_off);
  return launch_exact_conv(q, sx, codes, alpha_q, g, y, st);
}

// Output of a *_dfp layer call: fp32 (out_bits 0) or codes.
bool layer_out(int32_t out_bits, const float* out_scale, void* out, int64_t O, LayerOut* lo,
               fgq_status* err) {
  if (out_bits == 0) {
    *lo = LayerOut{static_cast<float*>(out), nullptr, nullptr, 0};
    return true;
  }
  if (out_bits != 8 && out_bits != 4) {
    *err = FGQ_ERR_BITS;
    return false;
  }
  if (out_bits == 4 && O % 2 != 0) {
    *err = FGQ_ERR_BITS;
    return false;
  }
  if (!out_scale) {
    *err = FGQ_ERR_NULL;
    return false;
  }
  *lo = LayerOut{nullptr, static_cast<uint8_t*>(out), out_scale, out_bits};
  return true;
}

}  // namespace

extern "C" {

const char* fgq_status_string(fgq_status s) {
  switch (s) {
    case FGQ_OK: return "FGQ_OK";
    case FGQ_ERR_NULL: return "FGQ_ERR_NULL: a required pointer is NULL";
    case FGQ_ERR_SHAPE: return "FGQ_ERR_SHAPE: invalid or inconsistent sizes";
    case FGQ_ERR_GROUP: return "FGQ_ERR_GROUP: group size must be >= 1 and divide C";
    case FGQ_ERR_BITS: return "FGQ_ERR_BITS: bits must be 8 or 4 (4 needs an even C or n)";
    case FGQ_ERR_NONFINITE: return "FGQ_ERR_NONFINITE: weights contain NaN or Inf";
    case FGQ_ERR_HIP: return "FGQ_ERR_HIP: HIP runtime error or no device";
    case FGQ_ERR_UNSUPPORTED: return "FGQ_ERR_UNSUPPORTED: method or shape not supported";
    case FGQ_ERR_WORKSPACE: return "FGQ_ERR_WORKSPACE: workspace missing or too small";
    case FGQ_ERR_RANGE: return "FGQ_ERR_RANGE: group scales too widely spread for the folded layout";
    default: return "FGQ: unknown status";
  }
}

int32_t fgq_abi_version(void) { return 2; }

fgq_status fgq_check_violations(int64_t* count, int32_t* first_site, int64_t* first_offset) {
#ifndef FGQ_CHECK
  (void)count, (void)first_site, (void)first_offset;
  return FGQ_ERR_UNSUPPORTED;
#else
  if (!count) return FGQ_ERR_NULL;
  if (hipDeviceSynchronize() != hipSuccess) return FGQ_ERR_HIP;
  std::vector<const void*> syms;
  {
    std::lock_guard<std::mutex> g(check_mutex());
    syms = check_records();
  }
  int64_t total = 0, offset = 0;
  int32_t site = 0;
  for (const void* sym : syms) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, sym) != hipSuccess) return FGQ_ERR_HIP;
    unsigned int rec[4];
    if (hipMemcpy(rec, p, sizeof rec, hipMemcpyDeviceToHost) != hipSuccess) return FGQ_ERR_HIP;
    if (rec[0] == 0) continue;
    if (site == 0) {
      site = static_cast<int32_t>(rec[1]);
      offset = static_cast<int64_t>(rec[2]) | (static_cast<int64_t>(rec[3]) << 32);
    }
    total += rec[0];
    if (hipMemset(p, 0, sizeof rec) != hipSuccess) return FGQ_ERR_HIP;
  }
  if (hipDeviceSynchronize() != hipSuccess) return FGQ_ERR_HIP;
  *count = total;
  if (first_site) *first_site = site;
  if (first_offset) *first_offset = offset;
  return FGQ_OK;
#endif
}

int32_t fgq_device_count(void) {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess) return 0;
  return n;
}

size_t fgq_codes_bytes(int64_t O, int64_t K) {
  if (O < 0 || K < 0) return 0;
  return static_cast<size_t>(O * ceil_div(K, 4));
}

int64_t fgq_group_count(int64_t O, int64_t K, int32_t G) {
  if (O < 0 || K < 0 || G < 1 || K % G != 0) return -1;
  return O * (K / G);
}

namespace {

// Wait for the offline step, then report non-finite weights (their groups
// carry alpha = NaN).
fgq_status ternarize_finish(const float* alpha, int64_t ng, hipStream_t st) {
  std::vector<float> host(static_cast<size_t>(ng));
  FGQ_TRY_HIP(hipMemcpyAsync(host.data(), alpha, sizeof(float) * ng, hipMemcpyDeviceToHost, st));
  FGQ_TRY_HIP(hipStreamSynchronize(st));
  for (int64_t i = 0; i < ng; ++i)
    if (host[i] != host[i]) return FGQ_ERR_NONFINITE;
  return FGQ_OK;
}

}  // namespace

fgq_status fgq_ternarize(const float* w, int64_t O, int64_t C, int32_t R, int32_t S, int32_t G,
                         int32_t method, uint8_t* codes, float* alpha, float* delta,
                         void* stream) {
  if (!w || !codes || !alpha) return FGQ_ERR_NULL;
  if (O < 1 || C < 1 || R < 1 || S < 1) return FGQ_ERR_SHAPE;
  if (G < 1 || C % G != 0) return FGQ_ERR_GROUP;
  if (method != FGQ_TERN_EXACT && method != FGQ_TERN_EXP_LEMMA && method != FGQ_TERN_GAUSS &&
      method != FGQ_TERN_KS)
    return FGQ_ERR_UNSUPPORTED;
  const int64_t K = static_cast<int64_t>(R) * S * C;
  hipStream_t st = as_stream(stream);
  if (method == FGQ_TERN_KS) {
    // the layer's rule by the K-S test, passed through alpha[0] (about to be
    // overwritten) to the host
    int32_t pick = 0;
    fgq_status rc = launch_ks(w, O * K, nullptr, reinterpret_cast<int32_t*>(alpha), st);
    if (rc != FGQ_OK) return rc;
    FGQ_TRY_HIP(hipMemcpyAsync(&pick, alpha, sizeof(pick), hipMemcpyDeviceToHost, st));
    FGQ_TRY_HIP(hipStreamSynchronize(st));
    method = pick;
  }
  fgq_status rc = launch_ternarize(w, O, C, R, S, G, method, codes, alpha, delta, nullptr, st);
  if (rc != FGQ_OK) return rc;
  return ternarize_finish(alpha, O * (K / G), st);
}

fgq_status fgq_ternarize_asym(const float* w, int64_t O, int64_t C, int32_t R, int32_t S, int32_t G,
                              uint8_t* codes, float* alpha, float* delta_p, float* delta_n, void* stream) {
  if (!w || !codes || !alpha) return FGQ_ERR_NULL;
  if (O < 1 || C < 1 || R < 1 || S < 1) return FGQ_ERR_SHAPE;
  if (G < 1 || C % G != 0) return FGQ_ERR_GROUP;
  const int64_t K = static_cast<int64_t>(R) * S * C;
  hipStream_t st = as_stream(stream);
  fgq_status rc = launch_ternarize(w, O, C, R, S, G, kTernAsym, codes, alpha, delta_p, delta_n, st);
  if (rc != FGQ_OK) return rc;
  return ternarize_finish(alpha, O * (K / G), st);
}

fgq_status fgq_ks_distances(const float* w, int64_t n, double* d, void* stream) {
  if (!w || !d) return FGQ_ERR_NULL;
  if (n < 1) return FGQ_ERR_SHAPE;
  return launch_ks(w, n, d, nullptr, as_stream(stream));
}

size_t fgq_quantize_ws_bytes(int64_t n) {
  if (n < 0) return 0;
  return sizeof(float) * static_cast<size_t>(quantize_partials(n));
}

fgq_status fgq_quantize_act(const float* x, int64_t n, int32_t bits, const float* scale_in,
                            uint8_t* q, float* scale_out, void* ws, size_t ws_bytes,
                            void* stream) {
  if (!x || !q || !scale_out) return FGQ_ERR_NULL;
  if (bits != 8 && bits != 4) return FGQ_ERR_BITS;
  if (n < 1) return FGQ_ERR_SHAPE;
  if (bits == 4 && n % 2 != 0) return FGQ_ERR_BITS;
  const int32_t np = quantize_partials(n);
  if (!scale_in && (!ws || ws_bytes < sizeof(float) * static_cast<size_t>(np)))
    return FGQ_ERR_WORKSPACE;
  return launch_quantize(x, n, bits, scale_in, q, scale_out, static_cast<float*>(ws), np,
                         as_stream(stream));
}

fgq_status fgq_quantize_act_noalloc(const float* x, int64_t n, int32_t bits, const float* scale_in,
                                    uint8_t* q, float* scale_out, void* stream) {
  if (!x || !q || !scale_out) return FGQ_ERR_NULL;
  if (bits != 8 && bits != 4) return FGQ_ERR_BITS;
  if (n < 1) return FGQ_ERR_SHAPE;
  if (bits == 4 && n % 2 != 0) return FGQ_ERR_BITS;
  const int32_t np = quantize_partials(n);
  if (np > kQuantScratchFloats) return FGQ_ERR_WORKSPACE;
  float* scratch = nullptr;
  if (!scale_in) {
    const fgq_status rc = quantize_scratch(&scratch);
    if (rc != FGQ_OK) return rc;
  }
  return launch_quantize(x, n, bits, scale_in, q, scale_out, scratch, np, as_stream(stream));
}

size_t fgq_prepared_bytes(int64_t O, int64_t K, int32_t G) {
  if (O < 1 || K < 1 || G < 1 || K % G != 0) return 0;
  return static_cast<size_t>(prepared_layout(O, K, G).total);
}

fgq_status fgq_prepare_weights(const uint8_t* codes, const float* alpha, int64_t O, int64_t K,
                               int32_t G, void* prepared, size_t prepared_bytes, void* stream) {
  if (!codes || !alpha || !prepared) return FGQ_ERR_NULL;
  if (O < 1 || K < 1) return FGQ_ERR_SHAPE;
  if (G < 1 || K % G != 0) return FGQ_ERR_GROUP;
  if (O > (1LL << 31) || K > (1LL << 31)) return FGQ_ERR_SHAPE;
  if (reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  const PreparedLayout L = prepared_layout(O, K, G);
  if (prepared_bytes < static_cast<size_t>(L.total)) return FGQ_ERR_WORKSPACE;
  hipStream_t st = as_stream(stream);
  fgq_status rc = launch_prepare(codes, alpha, O, K, G, prepared, st);
  if (rc != FGQ_OK || L.kind != kPrepFold) return rc;
  // The folded layout's accuracy guard: a channel whose scales do not fit
  // its fixed-point grid closely enough carries a NaN scale.
  std::vector<float> scale(static_cast<size_t>(O));
  FGQ_TRY_HIP(hipMemcpyAsync(scale.data(), static_cast<const char*>(prepared) + L.scale_off,
                             sizeof(float) * O, hipMemcpyDeviceToHost, st));
  FGQ_TRY_HIP(hipStreamSynchronize(st));
  for (int64_t o = 0; o < O; ++o)
    if (scale[o] != scale[o]) return FGQ_ERR_RANGE;
  return FGQ_OK;
}

fgq_status fgq_conv2d(const uint8_t* q, int32_t bits, const float* sx, int64_t B, int64_t H,
                      int64_t W, int64_t C, const uint8_t* codes, const float* alpha,
                      const void* prepared, int64_t O, int32_t R, int32_t S, int32_t stride_h,
                      int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t G, float* y,
                      void* stream) {
  if (!q || !sx || !codes || !alpha || !y) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(B, H, W, C, O, R, S, stride_h, stride_w, pad_h, pad_w, G, bits, &g, &err))
    return err;
  if (prepared && reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  return run_layer(q, sx, codes, alpha, prepared, g, LayerOut{y, nullptr, nullptr, 0}, stream);
}

fgq_status fgq_conv2d_residual(const uint8_t* q, int32_t bits, const float* sx, int64_t B, int64_t H,
                               int64_t W, int64_t C, const uint8_t* codes, const float* alpha,
                               const void* prepared, int64_t O, int32_t R, int32_t S, int32_t stride_h,
                               int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t G,
                               const float* res, float* y, void* stream) {
  if (!q || !sx || !codes || !alpha || !res || !y) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(B, H, W, C, O, R, S, stride_h, stride_w, pad_h, pad_w, G, bits, &g, &err))
    return err;
  if (prepared && reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  LayerOut lo{y, nullptr, nullptr, 2};
  lo.res = res;
  return run_layer(q, sx, codes, alpha, prepared, g, lo, stream);
}

fgq_status fgq_conv2d_residual_q(const uint8_t* q, int32_t bits, const float* sx, int64_t B, int64_t H,
                                 int64_t W, int64_t C, const uint8_t* codes, const float* alpha,
                                 const void* prepared, int64_t O, int32_t R, int32_t S, int32_t stride_h,
                                 int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t G,
                                 const float* res, float* y, int32_t out_bits, const float* out_scale,
                                 uint8_t* q_out, void* stream) {
  if (!q || !sx || !codes || !alpha || !res || !y || !out_scale || !q_out) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(B, H, W, C, O, R, S, stride_h, stride_w, pad_h, pad_w, G, bits, &g, &err))
    return err;
  if (out_bits != 8 && out_bits != 4) return FGQ_ERR_BITS;
  if (out_bits == 4 && O % 2 != 0) return FGQ_ERR_BITS;
  if (prepared && reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  LayerOut lo{y, q_out, out_scale, 2 | out_bits};
  lo.res = res;
  return run_layer(q, sx, codes, alpha, prepared, g, lo, stream);
}

fgq_status fgq_conv2d_q(const uint8_t* q, int32_t bits, const float* sx, int64_t B, int64_t H,
                        int64_t W, int64_t C, const uint8_t* codes, const float* alpha,
                        const void* prepared, int64_t O, int32_t R, int32_t S, int32_t stride_h,
                        int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t G, int32_t out_bits,
                        const float* out_scale, uint8_t* q_out, void* stream) {
  if (!q || !sx || !codes || !alpha || !out_scale || !q_out) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(B, H, W, C, O, R, S, stride_h, stride_w, pad_h, pad_w, G, bits, &g, &err))
    return err;
  if (out_bits != 8 && out_bits != 4) return FGQ_ERR_BITS;
  if (out_bits == 4 && O % 2 != 0) return FGQ_ERR_BITS;
  if (prepared && reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  return run_layer(q, sx, codes, alpha, prepared, g, LayerOut{nullptr, q_out, out_scale, out_bits}, stream);
}

fgq_status fgq_gemm(const uint8_t* q, int32_t bits, const float* sx, int64_t M, int64_t K,
                    const uint8_t* codes, const float* alpha, const void* prepared, int64_t O,
                    int32_t G, float* y, void* stream) {
  if (!q || !sx || !codes || !alpha || !y) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(1, M, 1, K, O, 1, 1, 1, 1, 0, 0, G, bits, &g, &err)) return err;
  if (prepared && reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  return run_layer(q, sx, codes, alpha, prepared, g, LayerOut{y, nullptr, nullptr, 0}, stream);
}

fgq_status fgq_gemm_q(const uint8_t* q, int32_t bits, const float* sx, int64_t M, int64_t K,
                      const uint8_t* codes, const float* alpha, const void* prepared, int64_t O,
                      int32_t G, int32_t out_bits, const float* out_scale, uint8_t* q_out,
                      void* stream) {
  if (!q || !sx || !codes || !alpha || !out_scale || !q_out) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(1, M, 1, K, O, 1, 1, 1, 1, 0, 0, G, bits, &g, &err)) return err;
  if (out_bits != 8 && out_bits != 4) return FGQ_ERR_BITS;
  if (out_bits == 4 && O % 2 != 0) return FGQ_ERR_BITS;
  if (prepared && reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  return run_layer(q, sx, codes, alpha, prepared, g, LayerOut{nullptr, q_out, out_scale, out_bits}, stream);
}

fgq_status fgq_dfp_alpha(const float* alpha, int64_t n, int32_t bits, int8_t* A, int32_t* fl,
                         void* stream) {
  if (!alpha || !A || !fl) return FGQ_ERR_NULL;
  if (bits != 8 && bits != 4) return FGQ_ERR_BITS;
  if (n < 1) return FGQ_ERR_SHAPE;
  hipStream_t st = as_stream(stream);
  fgq_status rc = launch_dfp_alpha(alpha, n, bits, A, fl, st);
  if (rc != FGQ_OK) return rc;
  int32_t host = 0;
  FGQ_TRY_HIP(hipMemcpyAsync(&host, fl, sizeof(host), hipMemcpyDeviceToHost, st));
  FGQ_TRY_HIP(hipStreamSynchronize(st));
  return host == INT32_MIN ? FGQ_ERR_NONFINITE : FGQ_OK;
}

size_t fgq_prepared_bytes_dfp(int64_t O, int64_t K, int32_t G) {
  if (O < 1 || K < 1 || G < 1 || K % G != 0) return 0;
  return static_cast<size_t>(prepared_layout_dfp(O, K, G).total);
}

fgq_status fgq_prepare_weights_dfp(const uint8_t* codes, const float* alpha, int64_t O, int64_t K,
                                   int32_t G, int32_t alpha_bits, void* prepared,
                                   size_t prepared_bytes, void* stream) {
  if (!codes || !alpha || !prepared) return FGQ_ERR_NULL;
  if (O < 1 || K < 1) return FGQ_ERR_SHAPE;
  if (G < 1 || K % G != 0) return FGQ_ERR_GROUP;
  if (alpha_bits != 8 && alpha_bits != 4) return FGQ_ERR_BITS;
  if (O > (1LL << 31) || K > (1LL << 31)) return FGQ_ERR_SHAPE;
  if (reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  if (prepared_bytes < static_cast<size_t>(prepared_layout_dfp(O, K, G).total)) return FGQ_ERR_WORKSPACE;
  hipStream_t st = as_stream(stream);
  fgq_status rc = launch_prepare_dfp(codes, alpha, O, K, G, alpha_bits, prepared, st);
  if (rc != FGQ_OK) return rc;
  int32_t host = 0;
  FGQ_TRY_HIP(hipMemcpyAsync(&host, prepared, sizeof(host), hipMemcpyDeviceToHost, st));
  FGQ_TRY_HIP(hipStreamSynchronize(st));
  return host == INT32_MIN ? FGQ_ERR_NONFINITE : FGQ_OK;
}

fgq_status fgq_conv2d_dfp(const uint8_t* q, int32_t bits, const float* sx, int64_t B, int64_t H,
                          int64_t W, int64_t C, const uint8_t* codes, const void* prepared,
                          int64_t O, int32_t R, int32_t S, int32_t stride_h, int32_t stride_w,
                          int32_t pad_h, int32_t pad_w, int32_t G, int32_t out_bits,
                          const float* out_scale, void* out, void* stream) {
  if (!q || !sx || !codes || !prepared || !out) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(B, H, W, C, O, R, S, stride_h, stride_w, pad_h, pad_w, G, bits, &g, &err))
    return err;
  LayerOut lo;
  if (!layer_out(out_bits, out_scale, out, O, &lo, &err)) return err;
  if (reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  return run_layer_dfp(q, sx, codes, prepared, g, lo, stream);
}

fgq_status fgq_conv2d_dfp_residual(const uint8_t* q, int32_t bits, const float* sx, int64_t B, int64_t H,
                                   int64_t W, int64_t C, const uint8_t* codes, const void* prepared,
                                   int64_t O, int32_t R, int32_t S, int32_t stride_h, int32_t stride_w,
                                   int32_t pad_h, int32_t pad_w, int32_t G, const float* res, float* y,
                                   int32_t out_bits, const float* out_scale, uint8_t* q_out, void* stream) {
  if (!q || !sx || !codes || !prepared || !res || !y) return FGQ_ERR_NULL;
  if (out_bits != 0 && (!out_scale || !q_out)) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(B, H, W, C, O, R, S, stride_h, stride_w, pad_h, pad_w, G, bits, &g, &err))
    return err;
  if (out_bits != 0 && out_bits != 8 && out_bits != 4) return FGQ_ERR_BITS;
  if (out_bits == 4 && O % 2 != 0) return FGQ_ERR_BITS;
  if (reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  LayerOut lo{y, out_bits ? q_out : nullptr, out_bits ? out_scale : nullptr, 2 | out_bits};
  lo.res = res;
  return run_layer_dfp(q, sx, codes, prepared, g, lo, stream);
}

fgq_status fgq_gemm_dfp(const uint8_t* q, int32_t bits, const float* sx, int64_t M, int64_t K,
                        const uint8_t* codes, const void* prepared, int64_t O, int32_t G,
                        int32_t out_bits, const float* out_scale, void* out, void* stream) {
  if (!q || !sx || !codes || !prepared || !out) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(1, M, 1, K, O, 1, 1, 1, 1, 0, 0, G, bits, &g, &err)) return err;
  LayerOut lo;
  if (!layer_out(out_bits, out_scale, out, O, &lo, &err)) return err;
  if (reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  return run_layer_dfp(q, sx, codes, prepared, g, lo, stream);
}

size_t fgq_gemm_ws_bytes(int64_t M, int64_t K, int64_t O, int32_t G, int32_t fixed_point) {
  if (M < 1 || K < 1 || O < 1 || G < 1 || K % G != 0 || K > kFoldMaxK) return 0;
  if (!fixed_point && prepared_layout(O, K, G).kind != kPrepFold) return 0;
  int32_t sps = 0;
  int32_t splits = splitk_splits(M, K, O, &sps);
  if (splits <= 1) splits = 0;
  if (dfpx_shape_ok(M, K, O, G)) splits = std::max(splits, dfpx_splits(M, K, O, G, &sps));
  return static_cast<size_t>(splits) * (fixed_point ? 1 : 3) * static_cast<size_t>(M * O) * 4;
}

fgq_status fgq_gemm_ws(const uint8_t* q, int32_t bits, const float* sx, int64_t M, int64_t K,
                       const uint8_t* codes, const float* alpha, const void* prepared, int64_t O,
                       int32_t G, int32_t out_bits, const float* out_scale, void* out, void* ws,
                       size_t ws_bytes, void* stream) {
  if (!q || !sx || !codes || !alpha || !out) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(1, M, 1, K, O, 1, 1, 1, 1, 0, 0, G, bits, &g, &err)) return err;
  LayerOut lo;
  if (!layer_out(out_bits, out_scale, out, O, &lo, &err)) return err;
  if (prepared && reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  if (prepared && prepared_layout(O, K, G).kind == kPrepFold && fold_supported(g, q)) {
    const bool ws_ok = ws && reinterpret_cast<uintptr_t>(ws) % 4 == 0 && ws_bytes >= fgq_gemm_ws_bytes(M, K, O, G, 0);
    if (dfpx_supported(g, q)) {  // weights read as codes + scale digits
      if (!ws_ok) return FGQ_ERR_WORKSPACE;
      return launch_foldx_splitk(q, sx, prepared, g, lo, static_cast<int32_t*>(ws), as_stream(stream));
    }
    int32_t sps = 0;
    const int32_t splits = splitk_splits(M, K, O, &sps);
    if (splits > 1) {
      if (!ws_ok) return FGQ_ERR_WORKSPACE;
      return launch_fold_splitk(q, sx, prepared, g, lo, splits, sps, static_cast<int32_t*>(ws),
                                as_stream(stream));
    }
  }
  return run_layer(q, sx, codes, alpha, prepared, g, lo, stream);
}

fgq_status fgq_gemm_dfp_ws(const uint8_t* q, int32_t bits, const float* sx, int64_t M, int64_t K,
                           const uint8_t* codes, const void* prepared, int64_t O, int32_t G,
                           int32_t out_bits, const float* out_scale, void* out, void* ws,
                           size_t ws_bytes, void* stream) {
  if (!q || !sx || !codes || !prepared || !out) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(1, M, 1, K, O, 1, 1, 1, 1, 0, 0, G, bits, &g, &err)) return err;
  LayerOut lo;
  if (!layer_out(out_bits, out_scale, out, O, &lo, &err)) return err;
  if (reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  const bool ws_ok = ws && reinterpret_cast<uintptr_t>(ws) % 4 == 0 && ws_bytes >= fgq_gemm_ws_bytes(M, K, O, G, 1);
  if (dfpx_supported(g, q)) {  // weights read as codes + scale codes
    if (!ws_ok) return FGQ_ERR_WORKSPACE;
    return launch_dfpx_splitk(q, sx, prepared, g, lo, static_cast<int32_t*>(ws), as_stream(stream));
  }
  if (fold_dfp_supported(g, q)) {
    int32_t sps = 0;
    const int32_t splits = splitk_splits(M, K, O, &sps);
    if (splits > 1) {
      if (!ws_ok) return FGQ_ERR_WORKSPACE;
      return launch_fold_dfp_splitk(q, sx, prepared, g, lo, splits, sps, static_cast<int32_t*>(ws),
                                    as_stream(stream));
    }
  }
  return run_layer_dfp(q, sx, codes, prepared, g, lo, stream);
}

size_t fgq_prepared_bytes_w8(int64_t O, int64_t C, int32_t R, int32_t S) {
  if (O < 1 || C < 1 || R < 1 || S < 1) return 0;
  return static_cast<size_t>(prepared_layout_dfp(O, C * R * S, static_cast<int32_t>(C)).total);
}

fgq_status fgq_prepare_weights_w8(const float* w, int64_t O, int64_t C, int32_t R, int32_t S,
                                  void* prepared, size_t prepared_bytes, void* stream) {
  if (!w || !prepared) return FGQ_ERR_NULL;
  if (O < 1 || C < 1 || R < 1 || S < 1) return FGQ_ERR_SHAPE;
  if (O > (1LL << 31) || C * R * S > (1LL << 31)) return FGQ_ERR_SHAPE;
  if (reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  if (prepared_bytes < fgq_prepared_bytes_w8(O, C, R, S)) return FGQ_ERR_WORKSPACE;
  hipStream_t st = as_stream(stream);
  fgq_status rc = launch_prepare_w8(w, O, C, R, S, prepared, st);
  if (rc != FGQ_OK) return rc;
  int32_t host = 0;
  FGQ_TRY_HIP(hipMemcpyAsync(&host, prepared, sizeof(host), hipMemcpyDeviceToHost, st));
  FGQ_TRY_HIP(hipStreamSynchronize(st));
  return host == INT32_MIN ? FGQ_ERR_NONFINITE : FGQ_OK;
}

fgq_status fgq_conv2d_w8(const uint8_t* q, int32_t bits, const float* sx, int64_t B, int64_t H,
                         int64_t W, int64_t C, const void* prepared, int64_t O, int32_t R,
                         int32_t S, int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                         int32_t out_bits, const float* out_scale, void* out, void* stream) {
  if (!q || !sx || !prepared || !out) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  // one group per tap (G = C): the layout does not depend on the grouping
  if (!conv_geom(B, H, W, C, O, R, S, stride_h, stride_w, pad_h, pad_w, static_cast<int32_t>(C), bits,
                 &g, &err))
    return err;
  LayerOut lo;
  if (!layer_out(out_bits, out_scale, out, O, &lo, &err)) return err;
  if (reinterpret_cast<uintptr_t>(prepared) % 256 != 0) return FGQ_ERR_WORKSPACE;
  if (!fold_dfp_supported(g, q)) return FGQ_ERR_UNSUPPORTED;
  return launch_fold_dfp_conv(q, sx, prepared, g, lo, as_stream(stream));
}

fgq_status fgq_group_sums(const uint8_t* q, int32_t bits, int64_t B, int64_t H, int64_t W,
                          int64_t C, const uint8_t* codes, int64_t O, int32_t R, int32_t S,
                          int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                          int32_t G, int64_t row0, int64_t nrows, int32_t* P, void* stream) {
  if (!q || !codes || !P) return FGQ_ERR_NULL;
  ConvGeom g;
  fgq_status err;
  if (!conv_geom(B, H, W, C, O, R, S, stride_h, stride_w, pad_h, pad_w, G, bits, &g, &err))
    return err;
  if (row0 < 0 || nrows < 0 || row0 + nrows > g.M) return FGQ_ERR_SHAPE;
  return launch_group_sums(q, codes, g, row0, nrows, P, as_stream(stream));
}

}  // extern "C"
