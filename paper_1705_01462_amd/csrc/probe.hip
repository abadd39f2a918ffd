// probe.hip -- measurement utility: the sustained rate of the int8 matrix
// instruction of the layer kernels (v_mfma_i32_32x32x32_i8), so that the
// benchmark can report kernels against a measured peak beside the published
// one.  Four independent accumulation chains per wave keep the matrix unit
// busy across the instruction's latency; two workgroups of four waves per
// compute unit put two waves on each SIMD.
#include "fgq_internal.h"

namespace fgq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256) void mfma_i8_probe_kernel(int32_t iters, int32_t* __restrict__ out) {
  const v4i a = {static_cast<int>(threadIdx.x), 0x01020304, 0x05060708, 0x090A0B0C};
  const v4i b = {static_cast<int>(blockIdx.x), 0x0D0E0F10, 0x11121314, 0x15161718};
  v16i acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = c + r;
  for (int32_t i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc[c], 0, 0, 0);
  }
  int32_t sum = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) sum += acc[c][r];
  out[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = sum;
}

}  // namespace
}  // namespace fgq

extern "C" fgq_status fgq_probe_mfma_i8(int32_t blocks, int32_t iters, int32_t* out, int64_t out_elems,
                                        void* stream) {
  if (!out) return FGQ_ERR_NULL;
  if (blocks < 1 || iters < 1 || out_elems < static_cast<int64_t>(blocks) * 256) return FGQ_ERR_SHAPE;
  hipLaunchKernelGGL(fgq::mfma_i8_probe_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0,
                     fgq::as_stream(stream), iters, out);
  return fgq::last_launch();
}
