// bufcheck.h -- the kernels' global-memory loads through buffer descriptors,
// and the bounds checks of a checking build.
//
// The kernels read through raw buffer descriptors whose extent is the size
// of the buffer (or of its region) being read.  The hardware returns zeros
// for a load whose vector offset lies past that extent, and the kernels use
// this for zero padding, but the scalar offset is not part of the check: a
// load whose vector offset is in range and whose scalar offset carries it
// past the end reads whatever follows the buffer.  Compiled with
// -DFGQ_CHECK (libfgq_check.so), every load made through these helpers
// tests exactly that case, and the checked stores test the element or byte
// range they write.  A violation is counted in a device record of the
// compilation unit (vector atomics) and the access is suppressed (the load
// returns zeros, the store is skipped), so a checking run reports a bad
// access instead of faulting; fgq_check_violations() reads and clears the
// records of every unit.  Without FGQ_CHECK the helpers are the plain loads
// and the store checks are constant true.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace fgq {

// Which access a reported violation came from (first one per record).
enum CheckSite : uint32_t {
  kSiteActs = 1,      // activation codes (implicit-GEMM gather, GEMM rows)
  kSitePlanes = 2,    // prepared int8 weight planes
  kSiteCodes = 3,     // 2-bit codes in an operand order
  kSiteScales = 4,    // per-group scale bytes or digits
  kSiteAlpha = 5,     // per-group fp32 scales of the per-group kernel
  kSiteBias = 6,      // per-plane offset terms
  kSitePartials = 7,  // partial maxima of the quantization
  kSiteStoreY = 8,    // layer outputs (fp32 or codes)
  kSiteStorePart = 9, // split-K int32 sums
  kSiteStoreQ = 10,   // quantized activation codes
};

#ifdef FGQ_CHECK
// Host side (api.hip): remembers the record of one compilation unit, by the
// address of its host-side stand-in, for fgq_check_violations().
void check_register(const void* symbol);

// [0] violations, [1] site of the first, [2], [3] its byte offset (low, high).
static __device__ __align__(16) unsigned int check_record[4];

namespace {
struct CheckRecordRegistrar {
  CheckRecordRegistrar() { check_register(reinterpret_cast<const void*>(&check_record)); }
};
CheckRecordRegistrar check_record_registrar;
}  // namespace

__device__ inline void check_report(uint32_t site, uint64_t at) {
  if (atomicAdd(&check_record[0], 1u) == 0u) {
    check_record[1] = site;
    check_record[2] = static_cast<uint32_t>(at);
    check_record[3] = static_cast<uint32_t>(at >> 32);
  }
}
#endif

// Whether a store of `width` elements (or bytes) at index `at` stays within
// `limit`; reported when it does not (checking builds only).
__device__ inline bool check_store(uint32_t site, int64_t at, int64_t width, int64_t limit) {
#ifdef FGQ_CHECK
  if (at < 0 || at + width > limit) {
    check_report(site, static_cast<uint64_t>(at));
    return false;
  }
#else
  (void)site, (void)at, (void)width, (void)limit;
#endif
  return true;
}

// A raw buffer descriptor and, in checking builds, its extent and site.
struct Buf {
  __amdgpu_buffer_rsrc_t r;
#ifdef FGQ_CHECK
  uint32_t bytes, site;
#endif
};

__device__ inline Buf make_buf(const void* p, int32_t bytes, uint32_t site, int flags) {
  Buf b;
  b.r = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, bytes, flags);
#ifdef FGQ_CHECK
  b.bytes = static_cast<uint32_t>(bytes);
  b.site = site;
#else
  (void)site;
#endif
  return b;
}

// True when the load is in range for the hardware's check (vector offset)
// but not once the scalar offset is added.
__device__ inline bool load_escapes(const Buf& b, uint32_t voff, uint32_t soff, uint32_t width) {
#ifdef FGQ_CHECK
  const uint64_t v = static_cast<uint64_t>(voff) + width;
  if (v <= b.bytes && v + soff > b.bytes) {
    check_report(b.site, static_cast<uint64_t>(voff) + soff);
    return true;
  }
#else
  (void)b, (void)voff, (void)soff, (void)width;
#endif
  return false;
}

typedef int bc_v2i __attribute__((ext_vector_type(2)));
typedef int bc_v4i __attribute__((ext_vector_type(4)));

__device__ inline bc_v4i buf_load_b128(const Buf& b, uint32_t voff, uint32_t soff) {
  if (load_escapes(b, voff, soff, 16)) return bc_v4i{0, 0, 0, 0};
  return __builtin_amdgcn_raw_buffer_load_b128(b.r, voff, soff, 0);
}
__device__ inline bc_v2i buf_load_b64(const Buf& b, uint32_t voff, uint32_t soff) {
  if (load_escapes(b, voff, soff, 8)) return bc_v2i{0, 0};
  return __builtin_amdgcn_raw_buffer_load_b64(b.r, voff, soff, 0);
}
__device__ inline uint32_t buf_load_b32(const Buf& b, uint32_t voff, uint32_t soff) {
  if (load_escapes(b, voff, soff, 4)) return 0u;
  return __builtin_amdgcn_raw_buffer_load_b32(b.r, voff, soff, 0);
}
__device__ inline uint16_t buf_load_b16(const Buf& b, uint32_t voff, uint32_t soff) {
  if (load_escapes(b, voff, soff, 2)) return 0;
  return __builtin_amdgcn_raw_buffer_load_b16(b.r, voff, soff, 0);
}
__device__ inline uint8_t buf_load_b8(const Buf& b, uint32_t voff, uint32_t soff) {
  if (load_escapes(b, voff, soff, 1)) return 0;
  return __builtin_amdgcn_raw_buffer_load_b8(b.r, voff, soff, 0);
}

}  // namespace fgq
