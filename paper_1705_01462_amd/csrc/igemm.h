// igemm.h -- pieces shared by the matrix-core implicit-GEMM convolution
// kernels (fold_kernel.h, group_kernel.h).
//
// Implicit GEMM: output row m = (b, ho, wo), reduction index
// k = (r*S + s)*C + c, so a 16-element piece of k (C % 16 == 0) is 16
// consecutive channels of one input pixel.  A workgroup stages kTM rows x
// 128 k of activations per step into LDS: each thread gathers kXP pieces
// with raw buffer loads (out-of-image pieces use an offset past the end of
// the buffer, which the hardware returns as zeros), and publishes them,
// offset or unpacked to int8, to a double-buffered LDS tile whose 16-byte
// slots are XOR-swizzled so that the publish and the 32-row fragment reads
// each touch every bank once per pass.
#pragma once

#include <atomic>
#include <type_traits>

#include "fgq_internal.h"

namespace fgq {
namespace ig {

typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kKT = 128;          // K per step
constexpr int kRowB = kKT;        // LDS bytes per activation row
constexpr int kSlots = kKT / 16;  // 16-byte k-slots per row
constexpr int kBufFlags = 0x00020000;  // raw buffer descriptor word 3 (gfx9)
constexpr uint32_t kOutOfRange = 0x80000000u;

// Geometry and activation operand of a launch (sizes fit in 32 bits; the
// launchers check this).
struct ActArgs {
  const uint8_t* q;
  int32_t M, K, O;
  int32_t H, W, C, R, S, Ho, Wo, sh, sw, ph, pw;
  int32_t q_bytes;
  int32_t n_otiles, n_mtiles;
};

// Unpack 16 four-bit values (8 bytes, element 2i in the low nibble) to 16
// bytes in element order.
__device__ inline v4i unpack_u4x16(uint32_t x0, uint32_t x1) {
  const uint32_t lo0 = x0 & 0x0F0F0F0Fu, hi0 = (x0 >> 4) & 0x0F0F0F0Fu;
  const uint32_t lo1 = x1 & 0x0F0F0F0Fu, hi1 = (x1 >> 4) & 0x0F0F0F0Fu;
  v4i r;
  r.x = static_cast<int>(__builtin_amdgcn_perm(hi0, lo0, 0x05010400u));
  r.y = static_cast<int>(__builtin_amdgcn_perm(hi0, lo0, 0x07030602u));
  r.z = static_cast<int>(__builtin_amdgcn_perm(hi1, lo1, 0x05010400u));
  r.w = static_cast<int>(__builtin_amdgcn_perm(hi1, lo1, 0x07030602u));
  return r;
}

// Hardware places workgroup i on XCD i % 8: give each XCD a contiguous run
// of logical tiles (neighbouring row tiles share halos in that XCD's L2).
__device__ inline int xcd_swizzle(int bid, int n) {
  const int x = bid % 8, qn = n / 8, rn = n % 8;
  return x * qn + (x < rn ? x : rn) + bid / 8;
}

// Byte offset of the 16-byte k-slot `slot` of activation row `row` in LDS.
// The slot is XOR-swizzled by row/2 so that 16 consecutive rows at one slot
// (a fragment read) and 2 rows x 8 slots (a publish) each cover all 64
// banks once.
__device__ inline int lds_off(int row, int slot) {
  return row * kRowB + 16 * (slot ^ ((row >> 1) & (kSlots - 1)));
}

// Activation staging of a kTM-row tile.  kSmallC: C < 128 (several taps per
// step); otherwise at most one tap boundary per step.  In-loop index
// arithmetic is 32-bit and incremental, and every bounds test is bitwise so
// that a step stays one basic block for the scheduler.
template <int kBits, int kTM, bool kSmallC>
struct ActStager {
  static constexpr int kPieces = kTM * kSlots;
  static constexpr int kXP = (kPieces + kThreads - 1) / kThreads;
  // Pieces past the tile (kTM*8 not a multiple of 256) go to spare rows
  // after the tile so that every LDS store is unconditional.
  static constexpr int kStage = (kTM + (kXP * kThreads - kPieces) / kSlots) * kRowB;
  typedef typename std::conditional<kBits == 8, v4i, v2i>::type raw_t;

  int rowbase[kXP], hi0[kXP], wi0[kXP], xlds[kXP];
  bool rowok[kXP];
  int tr, ts, tc, tk;
  raw_t xraw[kXP];
  Buf rs;

  // Piece p = tid + 256*i is row p/kSlots of the tile, k-slot
  // 16*(p%kSlots) = 16*(tid%kSlots) of every step; the tap state starts at
  // step ks0.
  __device__ void init(const ActArgs& a, int m0, int tid, int ks0 = 0) {
    rs = make_buf(a.q, a.q_bytes, kSiteActs, kBufFlags);
#pragma unroll
    for (int i = 0; i < kXP; ++i) {
      const int p = tid + kThreads * i;
      const int m = m0 + p / kSlots;
      rowok[i] = (p < kPieces) && (m < a.M);
      const int mm = rowok[i] ? m : 0;
      const int wo_ = mm % a.Wo;
      const int t = mm / a.Wo;
      const int ho = t % a.Ho;
      const int b = t / a.Ho;
      hi0[i] = ho * a.sh - a.ph;
      wi0[i] = wo_ * a.sw - a.pw;
      rowbase[i] = (b * a.H + hi0[i]) * a.W + wi0[i];
      xlds[i] = lds_off(p / kSlots, p % kSlots);
    }
    tk = 16 * (tid % kSlots) + ks0 * kKT;
    const int rsi = tk / a.C;
    tc = tk - rsi * a.C;
    ts = rsi % a.S;
    tr = rsi / a.S;
  }

  // Move the tap state (r, s, c) of this thread's k to the next step.
  __device__ void advance(const ActArgs& a) {
    tk += kKT;
    if constexpr (kSmallC) {
      const int t = ts + (tc + kKT) / a.C;
      tc = (tc + kKT) % a.C;
      tr += t / a.S;
      ts = t % a.S;
    } else {
      tc += kKT;
      const bool wrap = tc >= a.C;
      tc = wrap ? tc - a.C : tc;
      const int t = ts + (wrap ? 1 : 0);
      const bool wrap2 = t == a.S;
      ts = wrap2 ? 0 : t;
      tr += wrap2 ? 1 : 0;
    }
  }

  __device__ void load(const ActArgs& a) {
#pragma unroll
    for (int i = 0; i < kXP; ++i) {
      const int hi = hi0[i] + tr, wi = wi0[i] + ts;
      const bool ok = rowok[i] & (tk < a.K) & (static_cast<unsigned>(hi) < static_cast<unsigned>(a.H)) &
                      (static_cast<unsigned>(wi) < static_cast<unsigned>(a.W));
      const int e = (rowbase[i] + tr * a.W + ts) * a.C + tc;  // element offset
      if constexpr (kBits == 8) {
        const uint32_t off = ok ? static_cast<uint32_t>(e) : kOutOfRange;
        xraw[i] = buf_load_b128(rs, off, 0);
      } else {
        const uint32_t off = ok ? static_cast<uint32_t>(e) >> 1 : kOutOfRange;
        xraw[i] = buf_load_b64(rs, off, 0);
      }
    }
  }

  // Publish the loaded pieces to one LDS stage: uint8 bytes are XORed with
  // `mask8` (a per-kernel offset encoding; zero padding is encoded the same
  // way), uint4 pieces are unpacked to bytes 0..15.
  __device__ void store(unsigned char* base, uint32_t mask8) {
#pragma unroll
    for (int i = 0; i < kXP; ++i) {
      v4i v;
      if constexpr (kBits == 8) {
        const int x = static_cast<int>(mask8);
        v = xraw[i];
        v.x ^= x; v.y ^= x; v.z ^= x; v.w ^= x;
      } else {
        v = unpack_u4x16(static_cast<uint32_t>(xraw[i].x), static_cast<uint32_t>(xraw[i].y));
      }
      *reinterpret_cast<v4i*>(base + xlds[i]) = v;
    }
  }
};

// Activation staging for C = 4 or 8 (kC), e.g. a first layer whose three
// image channels are padded to 4: a 16-element piece spans 16/kC taps, and
// the kC channels of one tap are the only contiguous run, so each tap is
// loaded on its own (kC bytes, or kC/2 for 4-bit activations) with its own
// bounds test and the piece is assembled in registers.  Same interface and
// LDS layout as ActStager.
template <int kBits, int kTM, int kC>
struct ActStagerTinyC {
  static_assert(kC == 4 || kC == 8, "tiny-C staging is for C = 4 or 8");
  static constexpr int kPieces = kTM * kSlots;
  static constexpr int kXP = (kPieces + kThreads - 1) / kThreads;
  static constexpr int kStage = (kTM + (kXP * kThreads - kPieces) / kSlots) * kRowB;
  static constexpr int kSub = 16 / kC;  // taps per piece

  int rowbase[kXP], hi0[kXP], wi0[kXP], xlds[kXP];
  bool rowok[kXP];
  int tk;
  uint32_t part[kXP][kSub][kC * kBits / 32 > 0 ? kC * kBits / 32 : 1];
  Buf rs;

  __device__ void init(const ActArgs& a, int m0, int tid, int ks0 = 0) {
    rs = make_buf(a.q, a.q_bytes, kSiteActs, kBufFlags);
#pragma unroll
    for (int i = 0; i < kXP; ++i) {
      const int p = tid + kThreads * i;
      const int m = m0 + p / kSlots;
      rowok[i] = (p < kPieces) && (m < a.M);
      const int mm = rowok[i] ? m : 0;
      const int wo_ = mm % a.Wo;
      const int t = mm / a.Wo;
      const int ho = t % a.Ho;
      const int b = t / a.Ho;
      hi0[i] = ho * a.sh - a.ph;
      wi0[i] = wo_ * a.sw - a.pw;
      rowbase[i] = (b * a.H + hi0[i]) * a.W + wi0[i];
      xlds[i] = lds_off(p / kSlots, p % kSlots);
    }
    tk = 16 * (tid % kSlots) + ks0 * kKT;
  }

  __device__ void advance(const ActArgs&) { tk += kKT; }

  __device__ void load(const ActArgs& a) {
#pragma unroll
    for (int j = 0; j < kSub; ++j) {
      const int k = tk + j * kC;
      const int tap = k / kC;
      const int r = tap / a.S;
      const int t = tap - r * a.S;
#pragma unroll
      for (int i = 0; i < kXP; ++i) {
        const int hi = hi0[i] + r, wi = wi0[i] + t;
        const bool ok = rowok[i] & (k < a.K) & (static_cast<unsigned>(hi) < static_cast<unsigned>(a.H)) &
                        (static_cast<unsigned>(wi) < static_cast<unsigned>(a.W));
        const int e = (rowbase[i] + r * a.W + t) * kC;  // element offset of the tap
        if constexpr (kBits == 8 && kC == 4) {
          part[i][j][0] = buf_load_b32(rs, ok ? static_cast<uint32_t>(e) : kOutOfRange, 0);
        } else if constexpr (kBits == 8) {
          const v2i v = buf_load_b64(rs, ok ? static_cast<uint32_t>(e) : kOutOfRange, 0);
          part[i][j][0] = static_cast<uint32_t>(v.x);
          part[i][j][1] = static_cast<uint32_t>(v.y);
        } else if constexpr (kC == 4) {
          part[i][j][0] = buf_load_b16(rs, ok ? static_cast<uint32_t>(e) >> 1 : kOutOfRange, 0);
        } else {
          part[i][j][0] = buf_load_b32(rs, ok ? static_cast<uint32_t>(e) >> 1 : kOutOfRange, 0);
        }
      }
    }
  }

  __device__ void store(unsigned char* base, uint32_t mask8) {
#pragma unroll
    for (int i = 0; i < kXP; ++i) {
      v4i v;
      if constexpr (kBits == 8) {
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < kSub; ++j)
#pragma unroll
          for (int d = 0; d < kC / 4; ++d) w[j * (kC / 4) + d] = part[i][j][d] ^ mask8;
        v = v4i{static_cast<int>(w[0]), static_cast<int>(w[1]), static_cast<int>(w[2]), static_cast<int>(w[3])};
      } else if constexpr (kC == 4) {
        v = unpack_u4x16(part[i][0][0] | (part[i][1][0] << 16), part[i][2][0] | (part[i][3][0] << 16));
      } else {
        v = unpack_u4x16(part[i][0][0], part[i][1][0]);
      }
      *reinterpret_cast<v4i*>(base + xlds[i]) = v;
    }
  }
};

// kCM: how the reduction index maps onto taps.  0: C % 16 == 0, C >= 128
// (at most one tap boundary per step); 1: C % 16 == 0, C < 128; 4 / 8:
// C = 4 / 8 (tiny-C staging).
template <int kBits, int kTM, int kCM>
using StagerFor = typename std::conditional<
    (kCM <= 1), ActStager<kBits, kTM, kCM == 1>,
    ActStagerTinyC<kBits, kTM, (kCM == 4 || kCM == 8) ? kCM : 4>>::type;

// Fill the size fields of ActArgs from a validated geometry.
inline void fill_act_args(const ConvGeom& g, const uint8_t* q, ActArgs* a) {
  a->q = q;
  a->M = static_cast<int32_t>(g.M);
  a->K = static_cast<int32_t>(g.K);
  a->O = static_cast<int32_t>(g.O);
  a->H = static_cast<int32_t>(g.H);
  a->W = static_cast<int32_t>(g.W);
  a->C = static_cast<int32_t>(g.C);
  a->R = g.R;
  a->S = g.S;
  a->Ho = static_cast<int32_t>(g.Ho);
  a->Wo = static_cast<int32_t>(g.Wo);
  a->sh = g.sh;
  a->sw = g.sw;
  a->ph = g.ph;
  a->pw = g.pw;
  const int64_t in_elems = g.B * g.H * g.W * g.C;
  a->q_bytes = static_cast<int32_t>(g.bits == 8 ? in_elems : in_elems / 2);
  a->n_otiles = a->n_mtiles = 0;
}

// Size limits shared by the matrix-core kernels: 16-channel pieces (or the
// tiny-C staging when allowed), 32-bit element offsets, and an activation
// buffer aligned for its widest load.
inline bool igemm_shape_ok(const ConvGeom& g, const uint8_t* q, bool tiny_c = false) {
  const uintptr_t qa = reinterpret_cast<uintptr_t>(q);
  const int64_t in_elems = g.B * g.H * g.W * g.C;
  const bool c16 = g.C % 16 == 0;
  const bool ctiny = tiny_c && (g.C == 4 || g.C == 8);
  const uintptr_t align = c16 ? (g.bits == 8 ? 16 : 8) : static_cast<uintptr_t>(g.C * g.bits / 8);
  return (c16 || ctiny) && g.K < (1LL << 30) && qa % align == 0 && in_elems < (1LL << 31) &&
         g.M < (1LL << 31) && g.O < (1LL << 30);
}

// Compute units of the current device (cached per device; 256 if unknown).
// Host threads may call this concurrently (calls on distinct streams are
// thread-safe): the cache entries are atomics, and threads that race on the
// first call store the same value.
inline int device_cus() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

inline int c_mode(int64_t C) { return C % 16 == 0 ? (C >= kKT ? 0 : 1) : static_cast<int>(C); }

}  // namespace ig
}  // namespace fgq
