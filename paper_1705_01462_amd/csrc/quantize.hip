// quantize.hip -- activation quantization to unsigned 8 or 4 bits with one
// scale per tensor (Sec. 4: activations are quantized before each
// convolution).  Streaming, HBM-bound.
//
// Dynamic scale: pass 1 writes one partial maximum per block to the caller's
// workspace; pass 2 has every block reduce those partials (a few KB from
// L2) to the same s = max/qmax before quantizing its slice, so there are no
// atomics, no zero-initialised state and no host synchronisation.  Both
// passes issue all of a thread's loads before using any of them (pass 2
// also before the partials are reduced), so each costs about one memory
// round trip plus its bytes (a thread requests all of its partials at once:
// one loop load at a time cost a round trip each).  For uint8 codes from
// aligned buffers, pass 2 reads one contiguous kilobyte per wave-wide load
// and stores four codes per lane (quantize_coalesced_kernel: 6.3 -> 4.9 us
// on a 12.8 MB input to uint8); from unaligned buffers each pass-2 thread
// turns 16 (u8) or 32 (u4) consecutive values into codes byte by byte.
//
// The codes (qcode.h) use the correctly rounded quotient x/s from the
// reciprocal and one exact correction rather than the full division
// sequence, which made pass 2 compute-bound.
#include <mutex>

#include "fgq_internal.h"
#include "qcode.h"

// The quotient arithmetic below relies on each operation being rounded as
// written.
#pragma clang fp contract(off)

namespace fgq {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256;
constexpr int kMaxPartials = 1024;
constexpr int kP1Vec = 4;  // float4 loads per pass-1 thread and iteration

__device__ inline float block_max(float v, float* red) {
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  const int wid = threadIdx.x / 64, lane = threadIdx.x % 64;
  if (lane == 0) red[wid] = v;
  __syncthreads();
  float m = red[0];
#pragma unroll
  for (int i = 1; i < kThreads / 64; ++i) m = fmaxf(m, red[i]);
  return m;
}

// The largest of pass 1's partial maxima: every thread requests its (up to
// kMaxPartials / kThreads) partials at once through a range-checked buffer
// (reads past npart return 0, neutral for maxima of non-negative values),
// so the reduction costs one round trip, then one block reduction.
__device__ inline float partials_max(const float* partials, int32_t npart, float* red) {
  const Buf rs = make_buf(partials, 4 * npart, kSitePartials, 0x00020000);
  float p[kMaxPartials / kThreads];
#pragma unroll
  for (int u = 0; u < kMaxPartials / kThreads; ++u)
    p[u] = __uint_as_float(buf_load_b32(rs, 4 * (threadIdx.x + kThreads * u), 0));
  float m = 0.0f;
#pragma unroll
  for (int u = 0; u < kMaxPartials / kThreads; ++u) m = fmaxf(m, p[u]);
  return block_max(m, red);
}

// Pass 1.  Aligned input: block b reads the 1024-float4 chunks b, b + grid,
// ... (one chunk when the grid covers the input), lane l of wave w taking
// float4 number 256*i + 64*w + l of a chunk: the chunk-to-block mapping of
// quantize_coalesced_kernel, so a block reads 16 contiguous kilobytes where
// a grid-strided loop spread its loads over the whole input (measured
// faster on a 12.8 MB input; pass 2 still fetches its chunk from beyond L2).
template <bool kAligned>
__global__ __launch_bounds__(kThreads) void absmax_partial_kernel(
    const float* __restrict__ x, int64_t n, float* __restrict__ partials) {
  __shared__ float red[kThreads / 64];
  float m = 0.0f;  // max(max x, 0); fmaxf ignores NaN
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  if (kAligned) {
    const v4f* x4 = reinterpret_cast<const v4f*>(x);
    const int64_t n4 = n / 4;
    const int64_t nch = ceil_div(n4, static_cast<int64_t>(kThreads) * kP1Vec);
    for (int64_t c = blockIdx.x; c < nch; c += gridDim.x) {
      v4f v[kP1Vec];
#pragma unroll
      for (int u = 0; u < kP1Vec; ++u) {
        const int64_t i = c * kThreads * kP1Vec + static_cast<int64_t>(u) * kThreads + threadIdx.x;
        v[u] = i < n4 ? x4[i] : v4f{0.0f, 0.0f, 0.0f, 0.0f};
      }
#pragma unroll
      for (int u = 0; u < kP1Vec; ++u) m = fmaxf(m, fmaxf(fmaxf(v[u].x, v[u].y), fmaxf(v[u].z, v[u].w)));
    }
    for (int64_t i = n4 * 4 + tid; i < n; i += stride) m = fmaxf(m, x[i]);
  } else {
    for (int64_t i = tid; i < n; i += stride) m = fmaxf(m, x[i]);
  }
  m = block_max(m, red);
  if (threadIdx.x == 0) partials[blockIdx.x] = m;
}

template <int kBits, bool kAligned>
__global__ __launch_bounds__(kThreads) void quantize_kernel(
    const float* __restrict__ x, int64_t n, const float* __restrict__ scale_in,
    const float* __restrict__ partials, int32_t npart, uint8_t* __restrict__ q,
    float* __restrict__ scale_out) {
  __shared__ float red[kThreads / 64];
  constexpr float qmax = kBits == 8 ? 255.0f : 15.0f;
  constexpr int kPer = kBits == 8 ? 16 : 32;  // values per 16-byte store
  constexpr int kBytes = kPer * kBits / 8;    // output bytes per thread
  const int64_t nchunks = n / kPer;
  const int64_t ch = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;

  // 1. issue this thread's loads
  float v[kPer];
  const bool have = ch < nchunks;
  if (have) {
    if (kAligned) {
      const v4f* x4 = reinterpret_cast<const v4f*>(x + ch * kPer);
#pragma unroll
      for (int i = 0; i < kPer / 4; ++i) {
        const v4f t = __builtin_nontemporal_load(&x4[i]);
        v[4 * i] = t.x;
        v[4 * i + 1] = t.y;
        v[4 * i + 2] = t.z;
        v[4 * i + 3] = t.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < kPer; ++i) v[i] = x[ch * kPer + i];
    }
  }
  // 2. the scale, while those loads are in flight
  float s;
  if (scale_in) {
    s = *scale_in;
  } else {
    const float m = partials_max(partials, npart, red);
    s = m > 0.0f ? m / qmax : 1.0f;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *scale_out = s;

  // 3. quantize and store
  const QScale qs = make_qscale(s, kBits);
  with_rcp(qs, [&](auto rcp) {
    auto code = [&](float val) { return qcode<decltype(rcp)::value>(val, qs); };
    if (have) {
      uint32_t out[kBytes / 4];
#pragma unroll
      for (int wd = 0; wd < kBytes / 4; ++wd) {
        uint32_t word = 0;
        if (kBits == 8) {
#pragma unroll
          for (int b = 0; b < 4; ++b) word |= code(v[4 * wd + b]) << (8 * b);
        } else {
#pragma unroll
          for (int b = 0; b < 8; ++b) word |= code(v[8 * wd + b]) << (4 * b);
        }
        out[wd] = word;
      }
      uint8_t* dst = q + ch * kBytes;
      const int64_t nq = kBits == 8 ? n : n / 2;  // code bytes
      if (!check_store(kSiteStoreQ, ch * kBytes, kBytes, nq)) {
      } else if (kAligned) {
#pragma unroll
        for (int i = 0; i < kBytes / 16; ++i) {
          typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
          const u32x4 w = {out[4 * i], out[4 * i + 1], out[4 * i + 2], out[4 * i + 3]};
          __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(dst) + i);
        }
      } else {
#pragma unroll
        for (int i = 0; i < kBytes; ++i) dst[i] = static_cast<uint8_t>(out[i / 4] >> (8 * (i % 4)));
      }
    }
    // 4. the tail (fewer than kPer values), one byte per thread of the grid
    const int64_t done = nchunks * kPer;
    const int64_t tail_bytes = kBits == 8 ? (n - done) : (n - done) / 2;
    if (ch < tail_bytes) {
      if (kBits == 8) {
        if (check_store(kSiteStoreQ, done + ch, 1, n)) q[done + ch] = static_cast<uint8_t>(code(x[done + ch]));
      } else {
        const int64_t e = done + 2 * ch;
        if (check_store(kSiteStoreQ, e / 2, 1, n / 2))
          q[e / 2] = static_cast<uint8_t>(code(x[e]) | (code(x[e + 1]) << 4));
      }
    }
  });
}

// Pass 2 from 16-byte aligned x and q: each wave-wide load is one
// contiguous kilobyte of x (lane l takes float4 number 256*i + 64*w + l of
// the block's 1024, i = 0..3), and the codes of those four values are
// stored where they belong (4 bytes for uint8, 2 for uint4: a contiguous
// 256 or 128 bytes per wave-wide store).
template <int kBits>
__global__ __launch_bounds__(kThreads) void quantize_coalesced_kernel(
    const float* __restrict__ x, int64_t n, const float* __restrict__ scale_in,
    const float* __restrict__ partials, int32_t npart, uint8_t* __restrict__ q,
    float* __restrict__ scale_out) {
  __shared__ float red[kThreads / 64];
  constexpr int kVec = 4;  // float4 per thread
  const int64_t n4 = n / 4;
  const int64_t f0 = static_cast<int64_t>(blockIdx.x) * kThreads * kVec + threadIdx.x;
  const v4f* x4 = reinterpret_cast<const v4f*>(x);
  v4f v[kVec];
#pragma unroll
  for (int i = 0; i < kVec; ++i) {
    const int64_t f = f0 + static_cast<int64_t>(i) * kThreads;
    v[i] = f < n4 ? __builtin_nontemporal_load(&x4[f]) : v4f{0.0f, 0.0f, 0.0f, 0.0f};
  }
  float s;
  if (scale_in) {
    s = *scale_in;
  } else {
    const float m = partials_max(partials, npart, red);
    s = m > 0.0f ? m / (kBits == 8 ? 255.0f : 15.0f) : 1.0f;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *scale_out = s;
  const QScale qs = make_qscale(s, kBits);
  with_rcp(qs, [&](auto rcp) {
    auto code = [&](float val) { return qcode<decltype(rcp)::value>(val, qs); };
#pragma unroll
    for (int i = 0; i < kVec; ++i) {
      const int64_t f = f0 + static_cast<int64_t>(i) * kThreads;
      if (f < n4) {
        if constexpr (kBits == 8) {
          const uint32_t word = code(v[i].x) | (code(v[i].y) << 8) | (code(v[i].z) << 16) | (code(v[i].w) << 24);
          if (check_store(kSiteStoreQ, 4 * f, 4, n)) __builtin_nontemporal_store(word, reinterpret_cast<uint32_t*>(q) + f);
        } else {
          const uint32_t half = code(v[i].x) | (code(v[i].y) << 4) | (code(v[i].z) << 8) | (code(v[i].w) << 12);
          if (check_store(kSiteStoreQ, 2 * f, 2, n / 2))
            __builtin_nontemporal_store(static_cast<uint16_t>(half), reinterpret_cast<uint16_t*>(q) + f);
        }
      }
    }
    // the tail (n % 4 values; n is even for uint4), by the first block
    const int64_t done = n4 * 4;
    if (blockIdx.x == 0) {
      if (kBits == 8 && threadIdx.x < n - done && check_store(kSiteStoreQ, done + threadIdx.x, 1, n))
        q[done + threadIdx.x] = static_cast<uint8_t>(code(x[done + threadIdx.x]));
      if (kBits == 4 && threadIdx.x == 0 && n - done == 2 && check_store(kSiteStoreQ, done / 2, 1, n / 2))
        q[done / 2] = static_cast<uint8_t>(code(x[done]) | (code(x[done + 1]) << 4));
    }
  });
}

int64_t pass2_blocks(int64_t n, int32_t bits) {
  const int64_t per = bits == 8 ? 16 : 32;
  int64_t b = ceil_div(n / per, kThreads);
  if (b < 1) b = 1;  // the tail (< per values) needs at least one block
  return b;
}

}  // namespace

// The allocation-free entry point's scratch: pass 1's partial maxima (at
// most kMaxPartials floats for any n).  Each device holds its own copy at its
// own address; host code uses only the address from hipGetSymbolAddress,
// looked up once per device with that device current.
__device__ __align__(256) float scratch[kQuantScratchFloats];
static_assert(kQuantScratchFloats >= kMaxPartials, "scratch holds every partial");

fgq_status quantize_scratch(float** out) {
  static std::mutex mu;
  static float* ptr[kMaxDevices] = {};
  int dev = 0;
  FGQ_TRY_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return FGQ_ERR_HIP;
  std::lock_guard<std::mutex> lock(mu);
  if (!ptr[dev]) {
    void* p = nullptr;
    FGQ_TRY_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return FGQ_ERR_HIP;
    ptr[dev] = static_cast<float*>(p);
  }
  *out = ptr[dev];
  return FGQ_OK;
}

int32_t quantize_partials(int64_t n) {
  int64_t b = ceil_div(ceil_div(n, 4), static_cast<int64_t>(kThreads) * kP1Vec);
  if (b < 1) b = 1;
  if (b > kMaxPartials) b = kMaxPartials;
  return static_cast<int32_t>(b);
}

fgq_status launch_quantize(const float* x, int64_t n, int32_t bits,
                           const float* scale_in, uint8_t* q, float* scale_out,
                           float* partials, int32_t npart, hipStream_t st) {
  const bool aligned = (reinterpret_cast<uintptr_t>(x) % 16 == 0) &&
                       (reinterpret_cast<uintptr_t>(q) % 16 == 0);
  if (!scale_in) {
    if (aligned)
      hipLaunchKernelGGL(absmax_partial_kernel<true>, dim3(npart), dim3(kThreads), 0, st, x, n, partials);
    else
      hipLaunchKernelGGL(absmax_partial_kernel<false>, dim3(npart), dim3(kThreads), 0, st, x, n, partials);
    if (last_launch() != FGQ_OK) return FGQ_ERR_HIP;
  }
  if (aligned) {
    const int64_t bc = ceil_div(n / 4, static_cast<int64_t>(kThreads) * 4);
    if (bc > 0x7fffffffLL) return FGQ_ERR_SHAPE;
    const dim3 gc(static_cast<uint32_t>(bc < 1 ? 1 : bc));
    if (bits == 8)
      hipLaunchKernelGGL(quantize_coalesced_kernel<8>, gc, dim3(kThreads), 0, st, x, n, scale_in, partials, npart,
                         q, scale_out);
    else
      hipLaunchKernelGGL(quantize_coalesced_kernel<4>, gc, dim3(kThreads), 0, st, x, n, scale_in, partials, npart,
                         q, scale_out);
    return last_launch();
  }
  const int64_t blocks = pass2_blocks(n, bits);
  if (blocks > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  const dim3 grid(static_cast<uint32_t>(blocks));
  if (bits == 8)
    hipLaunchKernelGGL((quantize_kernel<8, false>), grid, dim3(kThreads), 0, st, x, n, scale_in, partials, npart, q,
                       scale_out);
  else
    hipLaunchKernelGGL((quantize_kernel<4, false>), grid, dim3(kThreads), 0, st, x, n, scale_in, partials, npart, q,
                       scale_out);
  return last_launch();
}

}  // namespace fgq
