// epilogue.h -- the output stores of the matrix-core layer kernels.
//
// After the K loop a wave holds kNB blocks of 32 rows x 32 channels in the
// 32x32 matrix-instruction layout: lane l owns channel l % 32 and, for
// accumulator r = 0..15, row 8*(r/4) + 4*(l/32) + r%4 of the block.  Stored
// straight from that layout, every store instruction writes 32 consecutive
// channels of two rows: 128-byte row pieces for fp32, 32 bytes for 8-bit
// codes, 16 for 4-bit codes.  The number of store instructions, not the
// bytes, then bounds the epilogue of a layer with a large output.
//
// The staged form therefore passes each block through LDS: for block c the
// four waves write their 32x32 pieces into one (kNWM * 32 rows) x (kTO
// channels) tile, and the workgroup then writes whole tile rows with 16-byte
// non-temporal stores (a wave writes a kilobyte of consecutive row bytes per
// instruction: 4x fewer instructions than fp32 stores from registers, 16x
// fewer than 8-bit ones).  It needs tile rows that start 16-byte aligned in
// the output (fp32: O % 4 == 0, 8-bit: O % 16 == 0, 4-bit: O % 32 == 0, and
// a 16-byte aligned output pointer); other shapes use the direct form.
//
// Output kinds (kOut, see qcode.h): 0 = fp32 y; 8 = one code per byte; 4 =
// two codes per byte, the even channel in the low nibble; 2 = fp32 y =
// max(v + res, 0), res an fp32 tensor of y's shape read at the same elements
// (a residual block's shortcut addition and ReLU fused into its last layer);
// 2 | 8 and 2 | 4 = that y and also its codes.  Codes follow qcode.h.
#pragma once

#include "qcode.h"

namespace fgq {
namespace ig {

template <int kOut, int kNWO>
struct EpiTile {
  static constexpr int kNWM = 4 / kNWO;
  static constexpr int kTO = 32 * kNWO;   // tile channels
  static constexpr int kRows = kNWM * 32;  // tile rows per block pass
  // the tile holds fp32 values when the kind writes fp32, else codes
  static constexpr int kRowBytes = out_f32(kOut) ? 4 * kTO : (out_code_bits(kOut) == 8 ? kTO : kTO / 2);
  // 8 extra dwords per row: the two rows one write instruction touches
  // (4 apart) start 32 dwords apart modulo 64, so with 64 LDS banks their
  // 32-dword pieces do not share a bank.
  static constexpr int kPitch = kRowBytes + 32;
  static constexpr int kBytes = kRows * kPitch;
  static constexpr int kChunksPerRow = kRowBytes / 16;
  static constexpr int kChunks = kRows * kChunksPerRow;
  static constexpr int kChanPerChunk = out_f32(kOut) ? 4 : (out_code_bits(kOut) == 8 ? 16 : 32);
};

// Host side: whether the staged form applies to an output of O channels
// (the fp32 output, its residual and its codes; pointers that are not used
// are null).  A staged fp32 chunk of 4 channels also carries their 4 (or 2)
// code bytes, which need 4- (or 2-) byte alignment.
inline bool epi_staged(int kind, int64_t O, const void* y, const void* q, const void* res = nullptr) {
  const auto al = [](const void* p, uintptr_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; };
  const int code_bits = kind == 1 ? 0 : (kind & 12);
  if (kind == 0 || (kind & 2))
    return O % 4 == 0 && al(y, 16) && al(res, 16) && al(q, code_bits == 4 ? 2 : 4);
  return O % (code_bits == 8 ? 16 : 32) == 0 && al(q, 16);
}


// The code of channel pair (o, o^1) as one byte, formed in the lane of the
// even channel (lanes l and l^1 hold channels o and o^1).
__device__ inline unsigned pair_nibbles(unsigned c) {
  const unsigned other = static_cast<unsigned>(__builtin_amdgcn_mov_dpp(static_cast<int>(c), 0xB1, 0xF, 0xF, false));
  return c | (other << 4);
}

struct OutPtrs {
  float* y;
  uint8_t* q;
  int M, O;
  const float* res;  // kinds with a residual
};

// Direct form: each lane stores its own values.  `val(c, r)` is the fp32
// output of block c, accumulator r; lanes of channels >= O store nothing.
template <int kOut, int kNB, bool kRcp, class Val>
__device__ inline void store_direct(const OutPtrs& out, const QScale& qs, int m_wave, int o, int lane, Val&& val) {
  constexpr int kCode = out_code_bits(kOut);
  if (o >= out.O) return;
#pragma unroll
  for (int c = 0; c < kNB; ++c) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m_wave + 32 * c + 8 * (r / 4) + 4 * (lane / 32) + (r % 4);
      if (m >= out.M) continue;
      const int64_t e = static_cast<int64_t>(m) * out.O + o;
      const int64_t n = static_cast<int64_t>(out.M) * out.O;
      float v = val(c, r);
      if constexpr (out_res(kOut)) {
        if (check_store(kSiteStoreY, e, 1, n)) v = add_relu(v, __builtin_nontemporal_load(out.res + e));
      }
      if constexpr (out_f32(kOut)) {
        if (check_store(kSiteStoreY, e, 1, n)) __builtin_nontemporal_store(v, out.y + e);
      }
      if constexpr (kCode == 8) {
        if (check_store(kSiteStoreY, e, 1, n))
          __builtin_nontemporal_store(static_cast<uint8_t>(qcode<kRcp>(v, qs)), out.q + e);
      } else if constexpr (kCode == 4) {
        const unsigned b = pair_nibbles(qcode<kRcp>(v, qs));
        if ((o & 1) == 0 && check_store(kSiteStoreY, e >> 1, 1, (n + 1) / 2))
          __builtin_nontemporal_store(static_cast<uint8_t>(b), out.q + (e >> 1));
      }
    }
  }
}

// Staged form (see above).  Every thread of the workgroup must call it;
// `lds` holds at least EpiTile<kOut, kNWO>::kBytes and is free on entry
// except for reads still in flight, which the first barrier waits for.
// m0 / ot0: the workgroup's first row and channel; wm / wo: the wave's row
// and channel position in the tile.
template <int kOut, int kNWO, int kNB, bool kRcp, class Val>
__device__ inline void store_staged(unsigned char* lds, const OutPtrs& out, const QScale& qs, int m0, int ot0,
                                    int wm, int wo, int tid, Val&& val) {
  using T = EpiTile<kOut, kNWO>;
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  constexpr bool kF32 = out_f32(kOut);
  constexpr int kCode = out_code_bits(kOut);
  const int lane = tid % 64;
  const int col = 32 * wo + lane % 32;  // the lane's channel within the tile
#pragma unroll
  for (int c = 0; c < kNB; ++c) {
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int lr = 32 * wm + 8 * (r / 4) + 4 * (lane / 32) + (r % 4);
      const float v = val(c, r);
      if constexpr (kF32) {
        *reinterpret_cast<float*>(lds + lr * T::kPitch + 4 * col) = v;
      } else if constexpr (kCode == 8) {
        lds[lr * T::kPitch + col] = static_cast<unsigned char>(qcode<kRcp>(v, qs));
      } else {
        const unsigned b = pair_nibbles(qcode<kRcp>(v, qs));
        if ((col & 1) == 0) lds[lr * T::kPitch + col / 2] = static_cast<unsigned char>(b);
      }
    }
    __syncthreads();
#pragma unroll
    for (int t0 = 0; t0 < T::kChunks; t0 += 256) {
      const int t = t0 + tid;
      if (T::kChunks % 256 != 0 && t >= T::kChunks) break;
      const int lr = t / T::kChunksPerRow, cb = t % T::kChunksPerRow;
      const int m = m0 + (lr / 32) * kNB * 32 + 32 * c + lr % 32;
      const int ch = ot0 + cb * T::kChanPerChunk;
      if (m < out.M && ch < out.O) {
        u32x4 w = *reinterpret_cast<const u32x4*>(lds + lr * T::kPitch + 16 * cb);
        const int64_t el = static_cast<int64_t>(m) * out.O + ch;  // the chunk's first element
        const int64_t n = static_cast<int64_t>(out.M) * out.O;
        if constexpr (kF32) {
          // four fp32 values of channels ch..ch+3: the residual and ReLU, the
          // fp32 store, and their codes
          const int64_t byte = 4 * el;
          if (check_store(kSiteStoreY, byte, 16, 4 * n)) {
            if constexpr (out_res(kOut)) {
              const u32x4 rv = __builtin_nontemporal_load(
                  reinterpret_cast<const u32x4*>(reinterpret_cast<const unsigned char*>(out.res) + byte));
#pragma unroll
              for (int i = 0; i < 4; ++i) w[i] = __float_as_uint(add_relu(__uint_as_float(w[i]), __uint_as_float(rv[i])));
            }
            __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(reinterpret_cast<unsigned char*>(out.y) + byte));
          }
          if constexpr (kCode == 8) {
            uint32_t cw = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) cw |= qcode<kRcp>(__uint_as_float(w[i]), qs) << (8 * i);
            if (check_store(kSiteStoreY, el, 4, n))
              __builtin_nontemporal_store(cw, reinterpret_cast<uint32_t*>(out.q + el));
          } else if constexpr (kCode == 4) {
            uint32_t cw = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) cw |= qcode<kRcp>(__uint_as_float(w[i]), qs) << (4 * i);
            if (check_store(kSiteStoreY, el / 2, 2, (n + 1) / 2))
              __builtin_nontemporal_store(static_cast<uint16_t>(cw), reinterpret_cast<uint16_t*>(out.q + el / 2));
          }
        } else {
          const int64_t byte = kCode == 8 ? el : el / 2;
          const int64_t nbytes = kCode == 8 ? n : n / 2;
          if (check_store(kSiteStoreY, byte, 16, nbytes))
            __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(out.q + byte));
        }
      }
    }
  }
}

}  // namespace ig
}  // namespace fgq
