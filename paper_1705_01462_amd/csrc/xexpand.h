// xexpand.h -- expansion of 2-bit ternary codes and per-group int8 scale
// bytes (a fixed-point scale code A, or one digit of a folded fp32 scale) to
// the int8 weights A*t of the matrix instruction's operand, in registers.
// Shared by the codes-expanding GEMM (dfpx.hip) and the convolution kernels
// (fold_kernel.h).
//
// Operand order (xlayout.h): lane l (channel 32*wave + l%32, half hf = l/32)
// holds, in 128-wide K step s and K quarter h, the 16 weights
// k = 128*s + 64*hf + 16*h + [0, 16); the activation fragment of the same
// lane reads the same 16 k of its row.  Within a quarter's 32 bits of codes
// byte b holds, at bits 2i, the code of weight 4i+b, so the permute selectors
// of weights 4i..4i+3 are (codes >> 2i) & 0x03030303.
#pragma once

#include "igemm.h"

namespace fgq {
namespace ig {

// Permute selectors of a quarter's 16 weights for the scale bytes' table:
// word i, byte b selects the int8 weight of weight 4i+b from the pair
// (-a, a) of scale-byte words (v_perm: selector j picks byte j of a, 4+j
// byte j of -a, 12 a zero byte).  The code c of each weight is turned into
// that selector by a first permute through the constant table
// [12, j, 12, 4+j] (code 0 -> zero, 1 -> +a_j, 3 -> -a_j; code 2 is never
// written), j being the scale byte of weights 4i..4i+3.  The selectors
// depend on the codes only, so the planes of one quarter share them.
template <int kG>
__device__ inline void selectors(uint32_t c32, uint32_t (&s)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t j = kG == 4 ? i : (kG == 8 ? i / 2 : 0);
    const uint32_t lut = 0x0Cu | (j << 8) | (0x0Cu << 16) | ((4u + j) << 24);
    s[i] = __builtin_amdgcn_perm(0u, lut, (c32 >> (2 * i)) & 0x03030303u);
  }
}

// The quarter's int8 weights for scale bytes a (A, or a digit of it, in
// [-127, 127]).  -a is formed four bytes at a time as ((a ^ 0x7F7F7F7F) +
// 0x01010101) ^ 0x80808080 (one's complement of a + 128, plus one, minus
// 128), with no carry between bytes because no byte is -128.
__device__ inline v4i expand16(const uint32_t (&s)[4], uint32_t a) {
  const uint32_t na = ((a ^ 0x7F7F7F7Fu) + 0x01010101u) ^ 0x80808080u;  // per byte: -a
  v4i w;
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = static_cast<int>(__builtin_amdgcn_perm(na, a, s[i]));
  return w;
}

// Scale-code bytes of one lane and step: 64/G of them (one for G >= 64).
template <int kG>
struct ACodes {
  static constexpr int kBytes = kG >= 64 ? 1 : 64 / kG;
  static constexpr int kWords = kBytes >= 4 ? kBytes / 4 : 1;
  uint32_t w[kWords];

  // off: per-lane byte offset; soff: a wave-uniform byte offset (not
  // covered by the buffer's range check).
  __device__ void load(const Buf& rs, int off, int soff = 0) {
    if constexpr (kBytes == 16) {
      const v4i v = buf_load_b128(rs, off, soff);
      for (int i = 0; i < 4; ++i) w[i] = static_cast<uint32_t>(v[i]);
    } else if constexpr (kBytes == 8) {
      const v2i v = buf_load_b64(rs, off, soff);
      w[0] = static_cast<uint32_t>(v.x);
      w[1] = static_cast<uint32_t>(v.y);
    } else if constexpr (kBytes == 4) {
      w[0] = buf_load_b32(rs, off, soff);
    } else if constexpr (kBytes == 2) {
      w[0] = buf_load_b16(rs, off, soff);
    } else {
      w[0] = buf_load_b8(rs, off, soff);
    }
  }
  // The A bytes of quarter h (16 weights), placed where expand16<kG> reads
  // them: four (G = 4), two (G = 8) or one (byte 0).
  __device__ uint32_t quarter(int h) const {
    if constexpr (kG == 4) return w[h];
    else if constexpr (kG == 8) return w[h / 2] >> (16 * (h % 2));
    else if constexpr (kG == 16) return w[0] >> (8 * h);
    else if constexpr (kG == 32) return w[0] >> (8 * (h / 2));
    else return w[0];
  }
};

// 16 ternary codes of one lane (32 bits, same byte and bit order) to the
// int8 weights t in {-1, 0, 1}: table [0, 1, 0, -1] indexed by the codes.
__device__ inline v4i expand_ternary16(uint32_t c32) {
  v4i w;
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = static_cast<int>(__builtin_amdgcn_perm(0u, 0xFF000100u, (c32 >> (2 * i)) & 0x03030303u));
  return w;
}

}  // namespace ig
}  // namespace fgq
