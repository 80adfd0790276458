// Internal interface between the C-ABI layer and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fp8q.h"

namespace fp8q {

struct QuantArgs {
  const uint16_t* x;  // bf16 bit patterns [rows][ldx]
  int64_t rows, cols, ldx;
  uint8_t* codes;     // [rows][ldc] or [cols][ldc] when transposed
  int64_t ldc;
  float* scales;
  int pow2;           // power-of-two scales (FP8Q_POW2_SCALE)
  int e5m2;           // E5M2 codes, F_max = 57344 (FP8Q_E5M2)
};

// granularity: the fp8q_granularity value; nscales: entries of `scales`.
hipError_t launch_quantize(const QuantArgs& a, int granularity, bool transposed, int64_t nscales,
                           hipStream_t s);
hipError_t launch_cast_f32(const float* x, int64_t n, float scale, bool e5m2, uint8_t* codes, hipStream_t s);

// Both backward-pass layouts from one read: `a` carries x and the 1x128
// output (codes [rows][ldc], scales [cols/128][rows]); codes_t / scales_t
// take the 128x1 output written transposed (codes [cols][ldc_t], scales
// [rows/128][cols]).
struct DualArgs {
  QuantArgs a;
  uint8_t* codes_t;
  int64_t ldc_t;
  float* scales_t;
};

hipError_t launch_quantize_dual(const DualArgs& d, hipStream_t s);

struct GemmArgs {
  const uint8_t* A;  // FP8 codes [M][lda] (E4M3, or E5M2 by the formats)
  const uint8_t* B;  // FP8 codes [N][ldb]
  const float* sA;
  const float* sB;
  uint16_t* C;       // bf16 [M][ldc]
  int64_t M, N, K, lda, ldb, ldc;
  // 1x128 scale layouts [K/128][rows]: distance between K blocks (the row
  // count of the whole operand, which a sub-problem may not span)
  int64_t sa_ld, sb_ld;
  // entries of sA / sB from their base pointers (reads past them are zero)
  int64_t sa_count, sb_count;
  // C and ldc allow 16-byte stores (else 8-byte)
  int c_aligned16;
  // quantized output (fp8q_gemm_quantized): E4M3 codes [M][ldq] and 1x128
  // scales [N/128][cs_ld] of the bf16 result (cs_ld: the whole problem's M)
  uint8_t* Cq;
  float* Cs;
  int64_t ldq, cs_ld;
  // split-K (fp8q_gemm_splitk): `splits` workgroups share a tile, each
  // summing a contiguous range of K blocks; their fp32 partial tiles go to
  // `part` and the last to arrive (counted in cnt[tile]) adds them up
  float* part = nullptr;
  uint32_t* cnt = nullptr;
  int splits = 1;
};

// kPairBlockE8: 1x128 x 128x128 with power-of-two scales (applied inside
// the matrix instruction)
enum GemmPair { kPairTensor = 0, kPairRow = 1, kPairBlock = 2, kPairBlockK = 3, kPairBlockE8 = 4 };

// formats: bit 0 = A's codes are E5M2, bit 1 = B's (kPairBlock and
// kPairBlockK only; 0 for E4M3 x E4M3).
hipError_t launch_gemm(const GemmArgs& g, int pair, int formats, hipStream_t s);

// Grouped GEMM: up to kMaxGroup problems of one pair (tensor, row or
// 1x128 x 128x128) and one K in one launch; tile_start is filled by the
// launcher (prefix sums of the tile counts).
constexpr int kMaxGroup = 8;
struct GemmGroup {
  GemmArgs prob[kMaxGroup];
  int tile_start[kMaxGroup + 1];
  int count;
};
// The same 32-bit offset limits as launch_gemm's sub-problems, per problem
// (else hipErrorInvalidValue; the C-ABI checks them first).
hipError_t launch_gemm_grouped(const GemmGroup& gs, int pair, hipStream_t s);
hipError_t launch_gemm_quantized(const GemmArgs& g, int pair, hipStream_t s);

// Split-K for skinny problems: the number of workgroups per 128 x 128 tile
// (1: no split, the call is launch_gemm's) and the workspace bytes it needs.
int gemm_splitk_splits(int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc);
int64_t gemm_splitk_workspace(int64_t M, int64_t N, int splits);
// g.part / g.cnt / g.splits set from a workspace of that size
hipError_t launch_gemm_splitk(const GemmArgs& g, int pair, hipStream_t s);

// Calibrated Clipping: per-token float32 arrays of n tokens, the grids
// l_min + k step (k < nl) and h_min + k step (k < nh), and a workspace of
// blocks x clip_slots(nl, nh) float64 partial sums (one block per `chunk`
// consecutive tokens).  The result goes to device memory.
constexpr int kClipMaxL = 24, kClipMaxH = 48;
constexpr int kClipMaxBlocks = 256;

struct ClipArgs {
  const float *adv, *w, *pi, *rb, *rf;
  int64_t n, chunk;
  int blocks, nl, nh;
  double c_low_ref, c_high_ref, l_min, h_min, step, inv_step, delta_l, delta_h, l_old, h_old;
  double* partials;
  fp8q_clip_result* result;
};

using ClipResult = fp8q_clip_result;

// float64 slots per block for these grid sizes (-1 when unsupported)
int clip_slots(int nl, int nh);
hipError_t launch_calibrate_clip(const ClipArgs& p, hipStream_t s);

// Bytes of the library's own partial-sum array for fp8q_calibrate_clip_noalloc:
// kClipMaxBlocks blocks of clip_slots(kClipMaxL, kClipMaxH) float64 sums.
constexpr int64_t kClipScratchBytes = FP8Q_CLIP_SCRATCH_BYTES;
// Device address of that array on the device of stream s (the current device
// for the null stream), looked up on the first call for each device.
hipError_t clip_scratch(hipStream_t s, double** ptr);

}  // namespace fp8q
