// xlayout.h -- the operand order of the codes-expanding GEMM (dfpx.hip),
// written at preparation time (dfp.hip for fixed-point scales, prepare.hip
// for the folded fp32 scales).
//
// Lane (channel o, half hf) of 128-wide K step ks holds k = 128*ks + 64*hf
// + [0, 64).  Regions are [O/128][Kp/128][4 waves][64 lanes][per-lane
// bytes], so that one wave-wide load is one contiguous block:
//   codes  16 bytes per lane; byte 4h+b holds, at bits 2i, the code of
//          k = 128*ks + 64*hf + 16h + 4i + b (a quarter's permute selectors
//          are then (word >> 2i) & 0x03030303);
//   scales xnb = dfpx_acode_bytes(G) bytes per lane; byte j is the int8
//          value (a scale code, or a digit of one) of the group holding
//          k = 128*ks + 64*hf + G*j (G = 128: of k = 128*ks).
#pragma once

#include "fgq_internal.h"

namespace fgq {

// Lane index (the per-lane byte offset divided by the per-lane size).
__device__ inline int64_t xfrag_lane(int64_t nk, int64_t o, int64_t ks, int hf) {
  return ((o / 128 * nk + ks) * 4 + (o % 128) / 32) * 64 + o % 32 + 32 * hf;
}

// The k whose group scale-code byte j of lane (ks, hf) holds.
__device__ inline int64_t xscale_k(int64_t ks, int hf, int j, int32_t G) {
  return G >= 128 ? 128 * ks : 128 * ks + 64 * hf + static_cast<int64_t>(G) * j;
}

// Block-cooperative: channel o's code region (zeros when !live); codes are
// the caller's 2-bit [O][ceil(K/4)] array.
__device__ inline void write_xcodes(const uint8_t* __restrict__ codes, int64_t o, int64_t K, int64_t Kp,
                                    bool live, uint8_t* __restrict__ xcodes) {
  const int64_t nk = Kp / 128, rb = ceil_div(K, 4);
  for (int64_t e = threadIdx.x; e < nk * 32; e += blockDim.x) {
    const int64_t ks = e / 32;
    const int hf = static_cast<int>((e % 32) / 16), B = static_cast<int>(e % 16);
    const int64_t k0 = 128 * ks + 64 * hf + 16 * (B / 4) + B % 4;
    uint32_t v = 0;
    if (live)
      for (int i = 0; i < 4; ++i) {
        const int64_t k = k0 + 4 * i;
        const uint32_t c = k < K ? (codes[o * rb + k / 4] >> (2 * (k % 4))) & 3u : 0u;
        v |= c << (2 * i);
      }
    xcodes[xfrag_lane(nk, o, ks, hf) * 16 + B] = static_cast<uint8_t>(v);
  }
}

}  // namespace fgq
