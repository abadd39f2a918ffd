// fold_kernel.h -- folded-scale FGQ layer on the int8 matrix cores (gfx950):
// the kernel template and its launch logic.  The output kind is a template
// parameter (fp32 y, or 8-/4-bit codes of the next layer's activations), and
// each kind is instantiated in a source file of its own (fold.hip,
// fold_q8.hip, fold_q4.hip; fold_dfp*.hip for fixed-point scales) so that
// they compile in parallel.
//
// With the per-group scales folded into three int8 digit planes (see
// prepare.hip), the layer is three exact int8 GEMMs sharing one activation
// operand:
//   S_j[o][m] = sum_k plane_j[o][k] * q'[m][k],   q' = q ^ 0x80 (uint8) or q (uint4)
//   y[m][o]   = sum_j (S_j + bias_j[o]) * (s_x * h_o * 255^j)
// The integer sums are exact (|S_j + bias_j| <= 255 * 127 * K < 2^31 for
// K <= 65536); the combination is three fp32 conversions and fused
// multiply-adds per output.  With fixed-point scales (kDfp, see dfp.hip)
// the scale is already in the single plane A*t, and the output is
// fp32(double(S) * (double(s_x) * 2^-fl)).
//
// Implicit GEMM: row m = (b, ho, wo), k = (r*S + s)*C + c, so a 16-element
// piece of k (C % 16 == 0) is 16 consecutive channels of one input pixel.
//
// Work split.  A 256-thread workgroup owns a tile of output rows x output
// channels and walks K in steps of 128 (four 32-wide K slices of the
// v_mfma_i32_32x32x32_i8 instruction, which runs at twice the rate of the
// 16x16x64 form on gfx950; the prepared K is padded to a multiple of 128
// with zero weights).  Its four waves are kNWO (channels) x 4/kNWO
// (rows); each wave owns 32 channels x kNB*32 rows, i.e. kNB 32x32 blocks
// per digit plane.
//  * Activations are the 32-row MFMA operand: gathered into LDS once per
//    workgroup per step (double-buffered, 128-byte rows with the 16-byte
//    slot XOR-swizzled by (row/2) % 8 so that both the row writes and the
//    32-row fragment reads hit every bank once per pass) and read by every
//    wave that shares those rows.
//  * Weights are the 32-column operand: raw buffer loads straight into
//    registers (every workgroup reads the same few hundred KB, so they come
//    from L2).  They are stored in fragment order, so each wave-wide load is
//    one contiguous kilobyte; a lane's offset is fixed and the K step is the
//    scalar offset, so the loop spends no vector instructions on them.
//  * Out-of-image activation pieces are loaded with an offset past the
//    buffer end, which the hardware returns as zeros (q = 0, then q' = -128
//    for uint8), so padding needs no select.
// The accumulators start at the per-plane bias (uint8), and the loads of
// step ks+1 are interleaved between the matrix instructions of step ks.
// A lane's 16 accumulators of a block are 16 rows of one channel; for each
// row the wave stores 32 consecutive channels (128 contiguous bytes).
// Workgroups are numbered so that consecutive row tiles land on one XCD
// (shared halos in that XCD's L2).  In-loop index arithmetic is 32-bit and
// incremental.
#pragma once

#include "igemm.h"
#include "epilogue.h"
#include "qcode.h"
#include "xexpand.h"

namespace fgq {

struct FoldArgs {
  ig::ActArgs x;
  const float* sx;
  const int8_t* planes;
  const int32_t* bias;
  const float* scale;
  float* y;
  uint8_t* qo;           // output codes (kOut 8 or 4)
  const float* oscale;   // their scale
  const float* res = nullptr;  // residual added before the ReLU (kOut 2)
  const int32_t* fl;     // fixed-point scales: fractional length (prepared header)
  int32_t* part;         // split K (kOut 1): int32 sums [splits][planes][M][O]
  int32_t splits, steps_per_split;  // K steps [split*sps, min(nk, (split+1)*sps)) per workgroup
  int32_t staged;        // epilogue through LDS (epi_staged)
  int32_t nks, planes_bytes;
  // Weights as stored (xg = 4 or 64; 0: the int8 planes above): 2-bit codes
  // and per-group int8 scale bytes (three digit planes, or the fixed-point
  // scale codes) in the operand order of xlayout.h, expanded in registers.
  int32_t xg;
  const uint8_t* xcodes;
  const int8_t* xdigits;
  int32_t xcodes_bytes, xdigits_bytes, xplane, nk128;
};

// The codes operand of a prepared buffer (fold or fixed-point layout, with
// `planes` scale bytes per group): used for G = 4 and G = 64, where the
// layout holds it; otherwise xg = 0 and the kernels read the int8 planes.
inline void set_codes_operand(FoldArgs& a, int32_t G, const char* base, const PreparedLayout& L, int planes) {
  a.xg = 0;
  const int64_t xnb = dfpx_acode_bytes(G);
  if ((G != 4 && G != 64) || xnb == 0) return;
  a.xg = G;
  a.xcodes = reinterpret_cast<const uint8_t*>(base + L.xcodes_off);
  a.xdigits = reinterpret_cast<const int8_t*>(base + L.xacodes_off);
  a.xcodes_bytes = static_cast<int32_t>(L.xacodes_off - L.xcodes_off);
  a.xdigits_bytes = static_cast<int32_t>(L.total - L.xacodes_off);
  a.xplane = planes > 1 ? static_cast<int32_t>(round_up(a.x.O, 128) * (L.Kp / 64) * xnb) : 0;
  a.nk128 = static_cast<int32_t>(L.Kp / 128);
}

// One launcher per output kind: kOut = 0 (fp32 y), 8 or 4 (codes).
fgq_status launch_fold_out_f32(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_out_q8(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_out_q4(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_out_res(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_out_res_q8(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_out_res_q4(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_dfp_out_f32(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_dfp_out_q8(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_dfp_out_q4(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_dfp_out_res(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_dfp_out_res_q8(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_dfp_out_res_q4(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_part(const FoldArgs& a, int bits, hipStream_t st);
fgq_status launch_fold_dfp_part(const FoldArgs& a, int bits, hipStream_t st);
// Short reductions (K <= 128) over many row tiles, fp32 group scales: the
// row-walking kernel of fold_rows.h, same results.
bool fold_rows_eligible(const FoldArgs& a);
fgq_status launch_fold_rows(const FoldArgs& a, int bits, int out_bits, hipStream_t st);

namespace {

using namespace ig;

template <int kBits, int kNWO, int kNB, int kCM, int kOut, bool kDfp, int kG>
__global__ __launch_bounds__(kThreads, kNB <= 2 ? 2 : 1) void fold_conv_kernel(FoldArgs a) {
  constexpr int kNWM = 4 / kNWO;
  constexpr int kTO = 32 * kNWO;
  constexpr int kTM = kNWM * kNB * 32;
  using Stager = StagerFor<kBits, kTM, kCM>;
  constexpr int kXP = Stager::kXP;
  constexpr int kStage = Stager::kStage;
  constexpr int kLds = 2 * kStage > EpiTile<kOut, kNWO>::kBytes ? 2 * kStage : EpiTile<kOut, kNWO>::kBytes;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLds];

  const int tid = threadIdx.x;
  const int lane = tid % 64, wave = tid / 64;
  const int wo = wave % kNWO, wm = wave / kNWO;
  // Workgroups of one K split are numbered together (they share activations).
  const int ntiles = a.x.n_otiles * a.x.n_mtiles;
  const int tsplit = xcd_swizzle(blockIdx.x, ntiles * a.splits);
  const int split = tsplit / ntiles, tile = tsplit % ntiles;
  const int o0 = (tile % a.x.n_otiles) * kTO + 32 * wo;  // this wave's first channel
  const int m0 = (tile / a.x.n_otiles) * kTM;             // workgroup's first row

  const Buf wrs = make_buf(a.planes, a.planes_bytes, kSitePlanes, kBufFlags);

  // ---- weight fragments: lane supplies channel o0 + lane%32, k-slot
  // 16*(lane/32) of K half h; the fragment-ordered planes put the wave's
  // 64 lanes x 16 bytes of (tile, step, plane, half) in one kilobyte.
  constexpr int kPlanes = kDfp ? 1 : 3;        // weight planes (fixed-point scales: one)
  constexpr int kTileB = kPlanes * 2 * 1024;   // bytes of one channel tile, one 64-wide K block
  const int wbase = (o0 / 32) * a.nks * kTileB + 16 * lane;

  const int nk_all = (a.x.K + kKT - 1) / kKT;
  const int ks0 = split * a.steps_per_split;  // this workgroup's K steps [ks0, nk)
  const int nk = ks0 + a.steps_per_split < nk_all ? ks0 + a.steps_per_split : nk_all;
  Stager xs;
  xs.init(a.x, m0, tid, ks0);

  // A step covers two 64-wide fragment blocks (K quarters hq = 2*blk + h).
  // The step is the scalar offset, which the buffer range check does not
  // cover, so a step past the last is clamped to the last one (those loads
  // are never used).
  // kG > 0: the codes (16 bytes per lane and step) and each plane's scale
  // bytes (64/G per lane and step) of the lane's channel, from the
  // 128-channel region of the operand order that holds it; the step is the
  // scalar offset (4 KB of codes, 256 * 64/G bytes of each plane).
  constexpr bool kX = kG > 0;
  using DW = ACodes<kX ? kG : 4>;
  constexpr int kAB = DW::kBytes;
  const int xl = ((o0 / 128) * a.nk128 * 4 + (o0 % 128) / 32) * 64 + lane;  // lane index at step 0
  const Buf crs = make_buf(a.xcodes, a.xcodes_bytes, kSiteCodes, kBufFlags);
  const Buf drs = make_buf(a.xdigits, a.xdigits_bytes, kSiteScales, kBufFlags);

  v4i wring[2][kX ? 1 : kPlanes][4];
  v4i cring[2];
  DW dring[2][kPlanes];
  auto load_w = [&](auto U, int ks) {
    constexpr int u = decltype(U)::value;
    ks = ks < nk ? ks : nk - 1;
    if constexpr (kX) {
      cring[u] = buf_load_b128(crs, 16 * xl, 4096 * ks);
#pragma unroll
      for (int j = 0; j < kPlanes; ++j) dring[u][j].load(drs, j * a.xplane + kAB * xl, 256 * kAB * ks);
    } else {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) {
        const int kso = (2 * ks + blk) * kTileB;
#pragma unroll
        for (int j = 0; j < kPlanes; ++j)
#pragma unroll
          for (int h = 0; h < 2; ++h)
            wring[u][j][2 * blk + h] =
                buf_load_b128(wrs, wbase + (2 * j + h) * 1024, kso);
      }
    }
  };

  // Accumulators start at the uint8 offset term 128 * sum_k plane_j[o][k]
  // of the lane's channel, so the epilogue needs no integer additions.
  v16i acc[kPlanes][kNB];
  {
    const int oc = o0 + lane % 32;
#pragma unroll
    for (int j = 0; j < kPlanes; ++j) {
      const int bj = (kBits == 8 && oc < a.x.O && ks0 == 0) ? a.bias[j * a.x.O + oc] : 0;
      v16i init;
#pragma unroll
      for (int r = 0; r < 16; ++r) init[r] = bj;
#pragma unroll
      for (int c = 0; c < kNB; ++c) acc[j][c] = init;
    }
  }

  // A-operand fragment addresses (row = wave rows + 32c + lane%32; slot
  // 2*quarter + lane/32 for the planes' fragment order, 4*(lane/32) +
  // quarter for the codes' operand order: the same 16 k as the lane's
  // weights, which is all the matrix instruction needs)
  int afrag[kNB][4];
#pragma unroll
  for (int c = 0; c < kNB; ++c)
#pragma unroll
    for (int h = 0; h < 4; ++h)
      afrag[c][h] = lds_off(wm * kNB * 32 + 32 * c + lane % 32, kX ? 4 * (lane / 32) + h : 2 * h + lane / 32);

  auto compute = [&](int stage, const v4i (&w)[kX ? 1 : kPlanes][4]) {
    const unsigned char* base = lds + stage * kStage;
    if constexpr (kNB <= 2) {
      // Two workgroups share the compute unit: read each K slice's
      // fragments just before use (fewer live registers); the other
      // workgroup's waves cover the LDS latency.
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        v4i xf[kNB];
#pragma unroll
        for (int c = 0; c < kNB; ++c) xf[c] = *reinterpret_cast<const v4i*>(base + afrag[c][h]);
#pragma unroll
        for (int c = 0; c < kNB; ++c)
#pragma unroll
          for (int j = 0; j < kPlanes; ++j)
            acc[j][c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xf[c], w[kX ? 0 : j][h], acc[j][c], 0, 0, 0);
      }
    } else {
      v4i xf[kNB][4];
#pragma unroll
      for (int c = 0; c < kNB; ++c)
#pragma unroll
        for (int h = 0; h < 4; ++h) xf[c][h] = *reinterpret_cast<const v4i*>(base + afrag[c][h]);
#pragma unroll
      for (int h = 0; h < 4; ++h)
#pragma unroll
        for (int c = 0; c < kNB; ++c)
#pragma unroll
          for (int j = 0; j < kPlanes; ++j)
            acc[j][c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xf[c][h], w[kX ? 0 : j][h], acc[j][c], 0, 0, 0);
    }
  };

  // The same with the weights expanded from codes and scale bytes, one K
  // quarter at a time: four permute selectors per quarter (shared by the
  // planes), then per plane the quarter's 16 int8 weights.  Software
  // pipelined: quarter h+1 is expanded (vector ALU) while quarter h's matrix
  // instructions run, so only quarter 0's expansion precedes them.
  auto expand_q = [&](int h, const v4i& cw, const DW (&dw)[kPlanes], v4i (&wq)[kPlanes]) {
    uint32_t sel[4];
    selectors<kX ? kG : 4>(static_cast<uint32_t>(cw[h]), sel);
#pragma unroll
    for (int j = 0; j < kPlanes; ++j) wq[j] = expand16(sel, dw[j].quarter(h));
  };
  auto compute_x = [&](int stage, const v4i& cw, const DW (&dw)[kPlanes]) {
    const unsigned char* base = lds + stage * kStage;
    v4i wq[2][kPlanes];
    v4i xf[2][kNB];
#pragma unroll
    for (int c = 0; c < kNB; ++c) xf[0][c] = *reinterpret_cast<const v4i*>(base + afrag[c][0]);
    expand_q(0, cw, dw, wq[0]);
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      if (h < 3) {
#pragma unroll
        for (int c = 0; c < kNB; ++c) xf[(h + 1) & 1][c] = *reinterpret_cast<const v4i*>(base + afrag[c][h + 1]);
        expand_q(h + 1, cw, dw, wq[(h + 1) & 1]);
      }
#pragma unroll
      for (int j = 0; j < kPlanes; ++j)
#pragma unroll
        for (int c = 0; c < kNB; ++c)
          acc[j][c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xf[h & 1][c], wq[h & 1][j], acc[j][c], 0, 0, 0);
    }
  };
  // Instruction order of a codes step (a hint to the scheduler, in groups):
  // the first quarter's fragment reads and expansion, then each quarter's
  // matrix instructions one at a time with the next quarter's expansion
  // and fragment reads between them, the weight prefetch loads among the
  // first quarter's.
  constexpr int kExpV = kX ? 11 + (kG == 4 ? 7 : 4) * kPlanes : 0;  // vector ops per quarter's expansion
  constexpr int kMq = kPlanes * kNB;                                   // matrix ops per quarter
  constexpr int kVper = (kExpV + kMq - 1) / (kMq > 0 ? kMq : 1);
  auto schedule_x = [&]() {
    __builtin_amdgcn_sched_group_barrier(0x100, kNB, 0);   // quarter 0 fragment reads
    __builtin_amdgcn_sched_group_barrier(0x002, kExpV, 0);  // quarter 0 expansion
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      if (h < 3) __builtin_amdgcn_sched_group_barrier(0x100, kNB, 0);  // next quarter's fragments
#pragma unroll
      for (int i = 0; i < kMq; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (h == 0 && i < 1 + kPlanes) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // weight prefetch
        if (h < 3) __builtin_amdgcn_sched_group_barrier(0x002, kVper, 0);
      }
    }
  };

  // Step ks: prefetch step ks+1 (weights into ring slot (ks+1)%2,
  // activations into registers), feed the matrix cores from LDS stage ks%2
  // and ring slot ks%2, then publish the prefetched activations to the
  // other LDS stage.  After the last step the prefetch repeats the last
  // step's weights (clamped) or reads nothing (activations), so the step has
  // no data-dependent branch; the loop is unrolled by 2 so that ring indices
  // are constants.
  auto step = [&](auto U, int ks) {
    constexpr int u = decltype(U)::value;
    // Activation loads first: the publish at the end of the step waits for
    // them, and the memory counter is in order, so weight loads issued
    // before them would be waited for too.
    xs.advance(a.x);
    xs.load(a.x);
    __builtin_amdgcn_sched_barrier(0);
    load_w(std::integral_constant<int, 1 - u>{}, ks + 1);
    if constexpr (kX) {
      compute_x(u, cring[u], dring[u]);
      schedule_x();
    } else {
      compute(u, wring[u]);
    }
    // Schedule: every fragment read first (distinct registers, LDS latency
    // paid once), then the matrix instructions with the weight prefetch
    // loads and their address arithmetic slotted between them, so the per-CU
    // load path works while the matrix cores do.
    if constexpr (kNB > 2) {
#pragma unroll
      for (int i = 0; i < 4 * kNB; ++i) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
      for (int i = 0; i < 4 * kPlanes; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 4 * kPlanes * kNB - 8 * kPlanes, 0);
    }
    __builtin_amdgcn_sched_barrier(0);  // the publish waits for the prefetch: keep it last
    xs.store(lds + (1 - u) * kStage, 0x80808080u);  // q - 128 (padding 0 -> -128)
    __syncthreads();
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  load_w(I0{}, ks0);
  xs.load(a.x);
  xs.store(lds, 0x80808080u);
  __syncthreads();
  int ks = ks0;
  for (; ks + 2 <= nk; ks += 2) {
    step(I0{}, ks);
    step(I1{}, ks + 1);
  }
  if (ks < nk) step(I0{}, ks);

  // ---- epilogue: lane holds rows m of channel o.
  const int o = o0 + lane % 32;
  if constexpr (kOut == 1) {
    // split K: this split's raw integer sums, [split][plane][m][o]
    int32_t* const part = a.part;
    const int M = a.x.M, O = a.x.O;
    if (o >= O) return;
#pragma unroll
    for (int j = 0; j < kPlanes; ++j)
#pragma unroll
      for (int c = 0; c < kNB; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + wm * kNB * 32 + 32 * c + 8 * (r / 4) + 4 * (lane / 32) + (r % 4);
          const int64_t e = (static_cast<int64_t>(split * kPlanes + j) * M + m) * O + o;
          if (m < M && check_store(kSiteStorePart, e, 1, static_cast<int64_t>(a.splits) * kPlanes * M * O))
            part[e] = acc[j][c][r];
        }
  } else {
    const float sx = *a.sx;
    // locals: a byte store may alias anything, including the argument block
    const OutPtrs out{a.y, a.qo, a.x.M, a.x.O, a.res};
    const bool staged = a.staged != 0;
    auto emit = [&](auto val) {
      with_out_scale<kOut>(a.oscale, [&](const QScale& qs, auto rcp) {
        constexpr bool kR = decltype(rcp)::value;
        if (staged)
          store_staged<kOut, kNWO, kNB, kR>(lds, out, qs, m0, o0 - 32 * wo, wm, wo, tid, val);
        else
          store_direct<kOut, kNB, kR>(out, qs, m0 + wm * kNB * 32, o, lane, val);
      });
    };
    if constexpr (kDfp) {
      // y = fp32(double(S) * (double(s_x) * 2^-fl)); the scale is exact.
      const int32_t fl = *a.fl;  // INT32_MIN marks rejected scales (never negated)
      const double cd = fl > -2048 && fl < 2048 ? static_cast<double>(sx) * ldexp(1.0, -fl) : 0.0;
      emit([&](int c, int r) { return static_cast<float>(static_cast<double>(acc[0][c][r]) * cd); });
    } else {
      const float c0 = o < a.x.O ? sx * a.scale[o] : 0.0f;
      const float c1 = c0 * 255.0f, c2 = c0 * 65025.0f;
      emit([&](int c, int r) {
        const float f2 = static_cast<float>(acc[2 % kPlanes][c][r]);
        const float f1 = static_cast<float>(acc[1 % kPlanes][c][r]);
        const float f0 = static_cast<float>(acc[0][c][r]);
        return fmaf(f2, c2, fmaf(f1, c1, f0 * c0));
      });
    }
  }
}

template <int kOut, bool kDfp, int kG, int kBits, int kNWO, int kNB>
fgq_status launch_cfg(const FoldArgs& a0, hipStream_t st) {
  constexpr int kTO = 32 * kNWO, kTM = (4 / kNWO) * kNB * 32;
  FoldArgs a = a0;
  a.x.n_otiles = (a.x.O + kTO - 1) / kTO;
  a.x.n_mtiles = (a.x.M + kTM - 1) / kTM;
  const int64_t n = static_cast<int64_t>(a.x.n_otiles) * a.x.n_mtiles * a.splits;
  if (n > 0x7fffffffLL) return FGQ_ERR_SHAPE;
  const dim3 grid(static_cast<uint32_t>(n));
  switch (c_mode(a.x.C)) {
    case 0: hipLaunchKernelGGL((fold_conv_kernel<kBits, kNWO, kNB, 0, kOut, kDfp, kG>), grid, dim3(kThreads), 0, st, a); break;
    case 1: hipLaunchKernelGGL((fold_conv_kernel<kBits, kNWO, kNB, 1, kOut, kDfp, kG>), grid, dim3(kThreads), 0, st, a); break;
    case 4:
      if constexpr (kG == 0 || kG == 4)
        hipLaunchKernelGGL((fold_conv_kernel<kBits, kNWO, kNB, 4, kOut, kDfp, kG>), grid, dim3(kThreads), 0, st, a);
      else
        return FGQ_ERR_UNSUPPORTED;  // a group of kG channels needs C >= kG
      break;
    default:
      if constexpr (kG == 0 || kG == 4)
        hipLaunchKernelGGL((fold_conv_kernel<kBits, kNWO, kNB, 8, kOut, kDfp, kG>), grid, dim3(kThreads), 0, st, a);
      else
        return FGQ_ERR_UNSUPPORTED;
      break;
  }
  return last_launch();
}

// Rows per wave: two 32-row blocks (kNB = 2) for every shape.  Measured on
// the benchmark and network layers, 32-row tiles (more weight traffic per
// matrix instruction) and 128-row tiles (one workgroup per compute unit,
// and register spills in the per-group kernel) were slower, and a tile
// count balance of ceil(tiles / CUs) * kNB never prefers kNB = 4 over 2.
// With weights expanded from codes at G = 4, 128-row waves fit without
// spills (accumulators in the 192 accumulation registers) and halve the
// expansion per matrix instruction, but a lone wave per SIMD leaves the
// load and LDS latencies exposed: slower on every ResNet-50 layer
// (1.0-1.55x).
template <int kOut, bool kDfp, int kG, int kBits, int kNWO>
fgq_status launch_nwo(const FoldArgs& a, hipStream_t st) {
  return launch_cfg<kOut, kDfp, kG, kBits, kNWO, 2>(a, st);
}

template <int kOut, bool kDfp, int kG, int kBits>
fgq_status launch_bits(const FoldArgs& a, hipStream_t st) {
  if (a.x.O > 64) return launch_nwo<kOut, kDfp, kG, kBits, 4>(a, st);
  if (a.x.O > 32) return launch_nwo<kOut, kDfp, kG, kBits, 2>(a, st);
  return launch_nwo<kOut, kDfp, kG, kBits, 1>(a, st);
}

template <int kOut, bool kDfp, int kG>
fgq_status launch_g(const FoldArgs& a, int bits, hipStream_t st) {
  return bits == 8 ? launch_bits<kOut, kDfp, kG, 8>(a, st) : launch_bits<kOut, kDfp, kG, 4>(a, st);
}

// Weights from codes for G = 4 and G = 64 (a.xg), else from the planes; the
// split-K partial kernels and the one-plane layer with fixed-point scales
// always read the planes (with one plane, the expansion's vector work
// outweighs the bytes it saves: 10.5 against 9.4 us on the 3x3 layer of
// 128 channels at 28x28, batch 32).
template <int kOut, bool kDfp = false>
fgq_status launch_out(const FoldArgs& a, int bits, hipStream_t st) {
  if constexpr (kOut != 1 && !kDfp) {
    if (a.xg == 4) return launch_g<kOut, kDfp, 4>(a, bits, st);
    if (a.xg == 64) return launch_g<kOut, kDfp, 64>(a, bits, st);
  }
  return launch_g<kOut, kDfp, 0>(a, bits, st);
}

}  // namespace
}  // namespace fgq
