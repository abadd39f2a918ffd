// fold_rows.h -- the folded-scale layer (fold_kernel.h, fp32 group scales in
// three int8 digit planes) for short reductions over many output rows: one
// 128-wide K step (K <= 128), more than 64 channels and at least two row
// tiles per workgroup, as in the 1x1 convolutions that widen 64 or 128
// channels of a residual network at large spatial sizes.
//
// The one-tile-per-workgroup kernel spends most of such a layer refetching
// the channel tile's weights: a 64-row tile has one K step of matrix work
// but loads the same 3 x 128 x 128 weight bytes (48 KB) as every other tile.
// Here a workgroup loads its channel tile's weights once, keeps them in
// registers (the weights stay live through the epilogue, which the register
// budget of two waves per SIMD allows for one step and four channel waves),
// and walks row tiles mt0, mt0 + stride, ... of that channel tile.  The next
// tile's activation loads are issued before the current tile's matrix work
// and output stores, so their latency is hidden behind them (the memory
// counter is in order: loads issued before the stores are waited for
// without waiting for the stores).
//
// With one weight plane (fixed-point scales) a tile's weights are 16 KB and
// the one-tile kernel, whose workgroups overlap on a compute unit, measured
// faster; those layers keep it.
//
// Arithmetic, operand layouts, accumulator start values and the epilogue are
// those of fold_conv_kernel, so the outputs are identical to it bit for bit.
#pragma once

#include "fold_kernel.h"

namespace fgq {
namespace {

using namespace ig;

template <int kBits, int kCM, int kOut>
__global__ __launch_bounds__(kThreads, 2) void fold_rows_kernel(FoldArgs a) {
  constexpr int kNWO = 4, kNB = 2, kPlanes = 3;
  constexpr int kTO = 32 * kNWO;  // 128 channels
  constexpr int kTM = kNB * 32;   // 64 rows
  using Stager = StagerFor<kBits, kTM, kCM>;
  constexpr int kLds = Stager::kStage > EpiTile<kOut, kNWO>::kBytes ? Stager::kStage : EpiTile<kOut, kNWO>::kBytes;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLds];

  const int tid = threadIdx.x;
  const int lane = tid % 64, wo = tid / 64;
  // channel tile fixed per workgroup; row tiles strided by the number of
  // workgroups per channel tile (the grid is a multiple of n_otiles)
  const int ot = blockIdx.x % a.x.n_otiles;
  const int mstride = gridDim.x / a.x.n_otiles;
  const int o0 = ot * kTO + 32 * wo;  // this wave's first channel
  const int o = o0 + lane % 32;       // the lane's channel

  // the step's weight fragments, as fold_conv_kernel loads them for step 0
  constexpr int kTileB = kPlanes * 2 * 1024;
  const Buf wrs = make_buf(a.planes, a.planes_bytes, kSitePlanes, kBufFlags);
  const int wbase = (o0 / 32) * a.nks * kTileB + 16 * lane;
  v4i w[kPlanes][4];
#pragma unroll
  for (int blk = 0; blk < 2; ++blk)
#pragma unroll
    for (int j = 0; j < kPlanes; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        w[j][2 * blk + h] = buf_load_b128(wrs, wbase + (2 * j + h) * 1024, blk * kTileB);

  int32_t bias[kPlanes];
#pragma unroll
  for (int j = 0; j < kPlanes; ++j) bias[j] = (kBits == 8 && o < a.x.O) ? a.bias[j * a.x.O + o] : 0;

  int afrag[kNB][4];
#pragma unroll
  for (int c = 0; c < kNB; ++c)
#pragma unroll
    for (int h = 0; h < 4; ++h) afrag[c][h] = lds_off(32 * c + lane % 32, 2 * h + lane / 32);

  const float c0 = o < a.x.O ? *a.sx * a.scale[o] : 0.0f;
  const float c1 = c0 * 255.0f, c2 = c0 * 65025.0f;
  const OutPtrs out{a.y, a.qo, a.x.M, a.x.O, a.res};
  const bool staged = a.staged != 0;

  int mt = blockIdx.x / a.x.n_otiles;
  Stager xs;
  if (mt < a.x.n_mtiles) {
    xs.init(a.x, mt * kTM, tid, 0);
    xs.load(a.x);
  }
  for (; mt < a.x.n_mtiles; mt += mstride) {
    const int m0 = mt * kTM;
    v16i acc[kPlanes][kNB];
#pragma unroll
    for (int j = 0; j < kPlanes; ++j) {
      v16i init;
#pragma unroll
      for (int r = 0; r < 16; ++r) init[r] = bias[j];
#pragma unroll
      for (int c = 0; c < kNB; ++c) acc[j][c] = init;
    }
    __syncthreads();  // the previous tile's LDS reads (fragments, staged epilogue) are done
    xs.store(lds, 0x80808080u);  // q - 128 (padding 0 -> -128)
    __syncthreads();
    if (mt + mstride < a.x.n_mtiles) {
      xs.init(a.x, m0 + mstride * kTM, tid, 0);
      xs.load(a.x);
    }
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      v4i xf[kNB];
#pragma unroll
      for (int c = 0; c < kNB; ++c) xf[c] = *reinterpret_cast<const v4i*>(lds + afrag[c][h]);
#pragma unroll
      for (int c = 0; c < kNB; ++c)
#pragma unroll
        for (int j = 0; j < kPlanes; ++j)
          acc[j][c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xf[c], w[j][h], acc[j][c], 0, 0, 0);
    }

    auto val = [&](int c, int r) {
      const float f2 = static_cast<float>(acc[2][c][r]);
      const float f1 = static_cast<float>(acc[1][c][r]);
      const float f0 = static_cast<float>(acc[0][c][r]);
      return fmaf(f2, c2, fmaf(f1, c1, f0 * c0));
    };
    with_out_scale<kOut>(a.oscale, [&](const QScale& qs, auto rcp) {
      constexpr bool kR = decltype(rcp)::value;
      if (staged)
        store_staged<kOut, kNWO, kNB, kR>(lds, out, qs, m0, ot * kTO, 0, wo, tid, val);
      else
        store_direct<kOut, kNB, kR>(out, qs, m0, o, lane, val);
    });
  }
}

template <int kOut, int kBits>
fgq_status launch_rows_bits(const FoldArgs& a0, hipStream_t st) {
  FoldArgs a = a0;
  a.x.n_otiles = (a.x.O + 127) / 128;
  a.x.n_mtiles = (a.x.M + 63) / 64;
  // two workgroups per compute unit, the same number for every channel tile
  const int64_t per_o = std::max<int64_t>(1, std::min<int64_t>(a.x.n_mtiles, 2LL * device_cus() / a.x.n_otiles));
  const int64_t n = per_o * a.x.n_otiles;
  if (n > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  const dim3 grid(static_cast<uint32_t>(n));
  if (c_mode(a.x.C) == 0)
    hipLaunchKernelGGL((fold_rows_kernel<kBits, 0, kOut>), grid, dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((fold_rows_kernel<kBits, 1, kOut>), grid, dim3(kThreads), 0, st, a);
  return last_launch();
}

template <int kOut>
fgq_status launch_rows(const FoldArgs& a, int bits, hipStream_t st) {
  return bits == 8 ? launch_rows_bits<kOut, 8>(a, st) : launch_rows_bits<kOut, 4>(a, st);
}

}  // namespace
}  // namespace fgq
