// splitk.hip -- split K for the folded kernels, for GEMMs (small M, large K:
// fully-connected layers at small batch) whose row and channel tiles alone
// would occupy few compute units.
//
// The K steps are divided among workgroups; each writes the raw int32 sums
// of its steps (for every plane, row and channel) to a caller-provided
// workspace [splits][planes][M][O], and one more kernel adds the splits in a
// fixed order and applies the folded kernel's own epilogue.  The integer
// totals are those of the unsplit kernel (every prefix of the sum stays
// within the int32 range of the unsplit accumulator), so the outputs are
// bit-identical to it; no atomics, and the workspace needs no clearing.
#include "fgq_internal.h"
#include "igemm.h"
#include "qcode.h"

#pragma clang fp contract(off)

namespace fgq {

int32_t splitk_splits(int64_t M, int64_t K, int64_t O, int32_t* steps_per_split) {
  const int64_t nk = ceil_div(K, 128);
  const int64_t nwo = O > 64 ? 4 : (O > 32 ? 2 : 1);
  const int64_t tiles = ceil_div(O, 32 * nwo) * ceil_div(M, (4 / nwo) * 64);
  const int64_t cus = ig::device_cus();
  *steps_per_split = static_cast<int32_t>(nk);
  if (nk < 4 || 2 * tiles >= cus) return 1;
  // enough workgroups for two per compute unit, at least two steps each, and
  // int32 sums (4 bytes per row and channel per split) within a quarter of
  // the weight bytes (one per weight per plane)
  int64_t splits = ceil_div(2 * cus, tiles);
  if (splits > nk / 2) splits = nk / 2;
  if (splits > K / (16 * M)) splits = K / (16 * M);
  if (splits < 2) return 1;
  const int64_t sps = ceil_div(nk, splits);
  *steps_per_split = static_cast<int32_t>(sps);
  return static_cast<int32_t>(ceil_div(nk, sps));
}

namespace {

template <int kOut, bool kDfp>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const int32_t* __restrict__ part, int32_t splits,
                                                            int32_t M, int32_t O, const float* __restrict__ sxp,
                                                            const float* __restrict__ scale,
                                                            const int32_t* __restrict__ flp, float* y,
                                                            uint8_t* qo, const float* oscale) {
  constexpr int kPlanes = kDfp ? 1 : 3;
  const int64_t n = static_cast<int64_t>(M) * O;
  const float sx = *sxp;
  double cd = 0.0;
  if constexpr (kDfp) {
    const int32_t fl = *flp;  // INT32_MIN marks rejected scales (never negated)
    cd = fl > -2048 && fl < 2048 ? static_cast<double>(sx) * ldexp(1.0, -fl) : 0.0;
  }
  with_out_scale<kOut>(oscale, [&](const QScale& qs, auto rcp) {
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; e < n;
         e += static_cast<int64_t>(gridDim.x) * 256) {
      const int o = static_cast<int>(e % O);
      int32_t S[kPlanes];
#pragma unroll
      for (int j = 0; j < kPlanes; ++j) S[j] = 0;
      for (int s = 0; s < splits; ++s)
#pragma unroll
        for (int j = 0; j < kPlanes; ++j) S[j] += part[static_cast<int64_t>(s * kPlanes + j) * n + e];
      float v;
      if constexpr (kDfp) {
        v = static_cast<float>(static_cast<double>(S[0]) * cd);
      } else {
        const float c0 = sx * scale[o];
        const float c1 = c0 * 255.0f, c2 = c0 * 65025.0f;
        v = fmaf(static_cast<float>(S[2 % kPlanes]), c2,
                 fmaf(static_cast<float>(S[1 % kPlanes]), c1, static_cast<float>(S[0]) * c0));
      }
      emit_out<kOut, decltype(rcp)::value>(y, qo, qs, e, n, o, v);
    }
  });
}

// Four consecutive elements per thread (O % 4 == 0, 16-byte aligned sums,
// output aligned to its 4-element piece): 16-byte loads of the sums, one
// store per thread.  Same arithmetic per element as splitk_reduce_kernel.
template <int kOut, bool kDfp>
__global__ __launch_bounds__(256) void splitk_reduce4_kernel(const int32_t* __restrict__ part, int32_t splits,
                                                             int32_t M, int32_t O, const float* __restrict__ sxp,
                                                             const float* __restrict__ scale,
                                                             const int32_t* __restrict__ flp, float* y,
                                                             uint8_t* qo, const float* oscale) {
  typedef int v4i __attribute__((ext_vector_type(4)));
  typedef float v4f __attribute__((ext_vector_type(4)));
  constexpr int kPlanes = kDfp ? 1 : 3;
  const int64_t n = static_cast<int64_t>(M) * O;
  const float sx = *sxp;
  double cd = 0.0;
  if constexpr (kDfp) {
    const int32_t fl = *flp;  // INT32_MIN marks rejected scales (never negated)
    cd = fl > -2048 && fl < 2048 ? static_cast<double>(sx) * ldexp(1.0, -fl) : 0.0;
  }
  with_out_scale<kOut>(oscale, [&](const QScale& qs, auto rcp) {
    for (int64_t e = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4; e < n;
         e += static_cast<int64_t>(gridDim.x) * 1024) {
      const int o = static_cast<int>(e % O);
      v4i S[kPlanes];
#pragma unroll
      for (int j = 0; j < kPlanes; ++j) S[j] = v4i{0, 0, 0, 0};
#pragma unroll 4
      for (int s = 0; s < splits; ++s)
#pragma unroll
        for (int j = 0; j < kPlanes; ++j)
          S[j] += *reinterpret_cast<const v4i*>(part + static_cast<int64_t>(s * kPlanes + j) * n + e);
      float v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (kDfp) {
          v[i] = static_cast<float>(static_cast<double>(S[0][i]) * cd);
        } else {
          const float c0 = sx * scale[o + i];
          const float c1 = c0 * 255.0f, c2 = c0 * 65025.0f;
          v[i] = fmaf(static_cast<float>(S[2 % kPlanes][i]), c2,
                      fmaf(static_cast<float>(S[1 % kPlanes][i]), c1, static_cast<float>(S[0][i]) * c0));
        }
      }
      if (!check_store(kSiteStoreY, e, 4, n)) continue;
      if constexpr (kOut == 0) {
        __builtin_nontemporal_store(v4f{v[0], v[1], v[2], v[3]}, reinterpret_cast<v4f*>(y + e));
      } else {
        constexpr bool kR = decltype(rcp)::value;
        const uint32_t c0 = qcode<kR>(v[0], qs), c1 = qcode<kR>(v[1], qs);
        const uint32_t c2 = qcode<kR>(v[2], qs), c3 = qcode<kR>(v[3], qs);
        if constexpr (kOut == 8)
          __builtin_nontemporal_store(c0 | (c1 << 8) | (c2 << 16) | (c3 << 24), reinterpret_cast<uint32_t*>(qo + e));
        else
          __builtin_nontemporal_store(static_cast<uint16_t>(c0 | (c1 << 4) | (c2 << 8) | (c3 << 12)),
                                      reinterpret_cast<uint16_t*>(qo + e / 2));
      }
    }
  });
}

template <bool kDfp>
fgq_status launch_reduce(const int32_t* part, int32_t splits, int64_t M, int64_t O, const float* sx,
                         const float* scale, const int32_t* fl, const LayerOut& out, hipStream_t st) {
  const int64_t n = M * O;
  const int32_t m = static_cast<int32_t>(M), o = static_cast<int32_t>(O);
  const uintptr_t out_align = out.bits == 0 ? 16 : (out.bits == 8 ? 4 : 2);
  const uintptr_t out_addr = out.bits == 0 ? reinterpret_cast<uintptr_t>(out.y) : reinterpret_cast<uintptr_t>(out.q);
  if (O % 4 == 0 && reinterpret_cast<uintptr_t>(part) % 16 == 0 && out_addr % out_align == 0) {
    const int64_t blocks4 = ceil_div(n, 1024) < 8192 ? ceil_div(n, 1024) : 8192;
    const dim3 grid4(static_cast<uint32_t>(blocks4));
    switch (out.bits) {
      case 0:
        hipLaunchKernelGGL((splitk_reduce4_kernel<0, kDfp>), grid4, dim3(256), 0, st, part, splits, m, o, sx, scale,
                           fl, out.y, out.q, out.scale);
        break;
      case 8:
        hipLaunchKernelGGL((splitk_reduce4_kernel<8, kDfp>), grid4, dim3(256), 0, st, part, splits, m, o, sx, scale,
                           fl, out.y, out.q, out.scale);
        break;
      default:
        hipLaunchKernelGGL((splitk_reduce4_kernel<4, kDfp>), grid4, dim3(256), 0, st, part, splits, m, o, sx, scale,
                           fl, out.y, out.q, out.scale);
        break;
    }
    return last_launch();
  }
  const int64_t blocks = ceil_div(n, 256) < 8192 ? ceil_div(n, 256) : 8192;
  const dim3 grid(static_cast<uint32_t>(blocks));
  switch (out.bits) {
    case 0:
      hipLaunchKernelGGL((splitk_reduce_kernel<0, kDfp>), grid, dim3(256), 0, st, part, splits, m, o, sx, scale, fl,
                         out.y, out.q, out.scale);
      break;
    case 8:
      hipLaunchKernelGGL((splitk_reduce_kernel<8, kDfp>), grid, dim3(256), 0, st, part, splits, m, o, sx, scale, fl,
                         out.y, out.q, out.scale);
      break;
    default:
      hipLaunchKernelGGL((splitk_reduce_kernel<4, kDfp>), grid, dim3(256), 0, st, part, splits, m, o, sx, scale, fl,
                         out.y, out.q, out.scale);
      break;
  }
  return last_launch();
}

}  // namespace

fgq_status launch_splitk_reduce(const int32_t* part, int32_t splits, bool dfp, int64_t M, int64_t O,
                                const float* sx, const float* scale, const int32_t* fl, const LayerOut& out,
                                hipStream_t st) {
  return dfp ? launch_reduce<true>(part, splits, M, O, sx, scale, fl, out, st)
             : launch_reduce<false>(part, splits, M, O, sx, scale, fl, out, st);
}

}  // namespace fgq
