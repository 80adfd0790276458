// Test driver for a host-only build of the C-ABI (abi.hip with the stub
// launchers of abi_stubs.cpp) under AddressSanitizer and
// UndefinedBehaviorSanitizer: every entry point with arguments that must be
// refused (null pointers, non-positive and absurdly large sizes, short
// leading dimensions, bad enums and flags, misalignment), which must return
// the documented status without reaching a launcher, and with valid
// arguments, which must reach exactly one launcher with the arguments the
// contract implies.  Pointers are never dereferenced (the launchers are
// stubs).  Exit status 0 when every check holds.
#include <stdint.h>
#include <stdio.h>

#include "fp8q.h"
#include "internal.h"

namespace fp8q {
extern int stub_calls;
extern int64_t stub_nscales;
extern GemmArgs stub_gemm;
extern int stub_pair;
}  // namespace fp8q

static int failures = 0;

#define EXPECT(call, want, launches)                                                                     \
  do {                                                                                                   \
    const int before = fp8q::stub_calls;                                                                 \
    const int got = (int)(call);                                                                         \
    if (got != (int)(want) || fp8q::stub_calls - before != (launches)) {                                 \
      fprintf(stderr, "line %d: %s -> %d (want %d), %d launches (want %d)\n", __LINE__, #call, got,      \
              (int)(want), fp8q::stub_calls - before, (launches));                                      \
      ++failures;                                                                                        \
    }                                                                                                    \
  } while (0)

template <typename T>
static T* fake(uintptr_t off = 0) {
  return reinterpret_cast<T*>(static_cast<uintptr_t>(0x10000) + off);
}

int main() {
  const int64_t BIG = INT64_MAX, HUGE_DIM = (int64_t)1 << 40;
  const uint8_t* cA = fake<const uint8_t>();
  const float* sA = fake<const float>();
  void* C = fake<void>();
  uint8_t* codes = fake<uint8_t>();
  float* scales = fake<float>();
  const void* x = fake<const void>();

  // scales_count
  EXPECT(fp8q_scales_count(256, 384, FP8Q_BLOCK_1x128, 0) == 768 ? 0 : 1, 0, 0);
  EXPECT(fp8q_scales_count(BIG, BIG, FP8Q_BLOCK_128x128, 0), -1, 0);
  EXPECT(fp8q_scales_count(256, HUGE_DIM, FP8Q_BLOCK_1x128, 1), -1, 0);
  EXPECT(fp8q_scales_count(-1, 128, FP8Q_ROW, 0), -1, 0);

  // quantize
  EXPECT(fp8q_quantize(x, 256, 384, 384, FP8Q_BLOCK_1x128, 0, codes, 384, scales, nullptr), FP8Q_OK, 1);
  EXPECT(fp8q::stub_nscales == 768 ? 0 : 1, 0, 0);
  EXPECT(fp8q_quantize(x, 256, 384, 384, FP8Q_BLOCK_1x128, FP8Q_OUT_TRANSPOSED, codes, 256, scales, nullptr),
         FP8Q_OK, 1);
  EXPECT(fp8q_quantize(nullptr, 256, 384, 384, FP8Q_BLOCK_1x128, 0, codes, 384, scales, nullptr), FP8Q_ERR_INVAL,
         0);
  EXPECT(fp8q_quantize(x, BIG, BIG, BIG, FP8Q_BLOCK_1x128, 0, codes, BIG, scales, nullptr),
         FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_quantize(x, 256, HUGE_DIM, HUGE_DIM, FP8Q_ROW, 0, codes, HUGE_DIM, scales, nullptr),
         FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_quantize(x, 256, 384, 383, FP8Q_ROW, 0, codes, 384, scales, nullptr), FP8Q_ERR_INVAL, 0);
  EXPECT(fp8q_quantize(x, 256, 384, 384, (fp8q_granularity)9, 0, codes, 384, scales, nullptr), FP8Q_ERR_INVAL, 0);
  EXPECT(fp8q_quantize(x, 256, 384, 384, FP8Q_ROW, 64, codes, 384, scales, nullptr), FP8Q_ERR_INVAL, 0);
  EXPECT(fp8q_quantize(x, 256, 200, 208, FP8Q_BLOCK_1x128, 0, codes, 208, scales, nullptr), FP8Q_ERR_UNSUPPORTED,
         0);
  EXPECT(fp8q_quantize(fake<const void>(2), 256, 384, 384, FP8Q_ROW, 0, codes, 384, scales, nullptr),
         FP8Q_ERR_ALIGN, 0);

  // dual
  EXPECT(fp8q_quantize_dual(x, 256, 384, 384, 0, codes, 384, scales, codes, 256, scales, nullptr), FP8Q_OK, 1);
  EXPECT(fp8q_quantize_dual(x, BIG, BIG, BIG, 0, codes, BIG, scales, codes, BIG, scales, nullptr),
         FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_quantize_dual(x, 256, 384, 384, 1, codes, 384, scales, codes, 256, scales, nullptr), FP8Q_ERR_INVAL,
         0);

  // GEMM
  EXPECT(fp8q_gemm(cA, sA, FP8Q_BLOCK_1x128, 4096, cA, sA, FP8Q_BLOCK_128x128, 4096, 16384, 12288, 4096, C, 12288,
                   nullptr),
         FP8Q_OK, 1);
  EXPECT(fp8q::stub_gemm.sa_count == 16384 * 32 && fp8q::stub_gemm.sb_count == 96 * 32 &&
                 fp8q::stub_pair == fp8q::kPairBlock
             ? 0
             : 1,
         0, 0);
  EXPECT(fp8q_gemm(cA, sA, FP8Q_TENSOR, 256, cA, sA, FP8Q_TENSOR, 256, 128, 256, 256, C, 256, nullptr), FP8Q_OK,
         1);
  EXPECT(fp8q_gemm(cA, sA, FP8Q_BLOCK_1x128, BIG, cA, sA, FP8Q_BLOCK_128x128, BIG, BIG, BIG, 4096, C, BIG, nullptr),
         FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_gemm(cA, sA, FP8Q_ROW, 4096, cA, sA, FP8Q_ROW, 4096, HUGE_DIM, 128, 4096, C, 128, nullptr),
         FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_gemm(cA, sA, FP8Q_BLOCK_1x128, 4096, cA, sA, FP8Q_ROW, 4096, 256, 256, 4096, C, 256, nullptr),
         FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_gemm(cA, sA, FP8Q_BLOCK_1x128, 4096, cA, sA, FP8Q_BLOCK_128x128, 4096, 0, 256, 4096, C, 256, nullptr),
         FP8Q_ERR_INVAL, 0);
  EXPECT(fp8q_gemm(cA, sA, FP8Q_BLOCK_1x128, 4096, cA, sA, FP8Q_BLOCK_128x128, 4096, 256, 256, 4000, C, 256,
                   nullptr),
         FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_gemm(fake<const uint8_t>(8), sA, FP8Q_BLOCK_1x128, 4096, cA, sA, FP8Q_BLOCK_128x128, 4096, 256, 256,
                   4096, C, 256, nullptr),
         FP8Q_ERR_ALIGN, 0);
  EXPECT(fp8q_gemm_formats(cA, sA, FP8Q_BLOCK_1x128, 4096, cA, sA, FP8Q_BLOCK_128x128, 4096, 256, 256, 4096, 3, C,
                           256, nullptr),
         FP8Q_OK, 1);
  EXPECT(fp8q_gemm_formats(cA, sA, FP8Q_ROW, 4096, cA, sA, FP8Q_ROW, 4096, 256, 256, 4096, 1, C, 256, nullptr),
         FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_gemm_pow2(cA, sA, FP8Q_BLOCK_1x128, 4096, cA, sA, FP8Q_BLOCK_128x128, 4096, 256, 256, 4096, C, 256,
                        nullptr),
         FP8Q_OK, 1);
  EXPECT(fp8q_gemm_pow2(cA, sA, FP8Q_BLOCK_1x128, BIG, cA, sA, FP8Q_BLOCK_128x128, BIG, BIG, BIG, 4096, C, BIG,
                        nullptr),
         FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_gemm_quantized(cA, sA, FP8Q_BLOCK_1x128, 4096, cA, sA, FP8Q_BLOCK_128x128, 4096, 256, 256, 4096,
                             codes, 256, scales, nullptr),
         FP8Q_OK, 1);
  EXPECT(fp8q_gemm_quantized(cA, sA, FP8Q_BLOCK_1x128, BIG, cA, sA, FP8Q_BLOCK_128x128, BIG, BIG, BIG, 4096,
                             codes, BIG, scales, nullptr),
         FP8Q_ERR_UNSUPPORTED, 0);

  // split-K: sizes, the split count and where the counters and partials go
  {
    const int64_t ws_down = fp8q_gemm_splitk_workspace(256, 4096, 12288);
    if (ws_down != 256 + 64 * 4 * 65536) {
      fprintf(stderr, "split-K workspace %lld\n", (long long)ws_down);
      ++failures;
    }
    EXPECT(fp8q_gemm_splitk_workspace(256, 12288, 4096), 0, 0);
    EXPECT(fp8q_gemm_splitk_workspace(0x7fffffff, 0x7fffffff, 0x7fffff80), 0, 0);
    EXPECT(fp8q_gemm_splitk_workspace(BIG, BIG, BIG), -1, 0);
    EXPECT(fp8q_gemm_splitk_workspace(0, 128, 1024), -1, 0);
    EXPECT(fp8q_gemm_splitk_workspace(HUGE_DIM, 128, 1024), -1, 0);
    uint8_t* ws = fake<uint8_t>(1 << 20);
    EXPECT(fp8q_gemm_splitk(cA, sA, FP8Q_BLOCK_1x128, 12288, cA, sA, FP8Q_BLOCK_128x128, 12288, 256, 4096, 12288, C,
                            4096, ws, ws_down, nullptr),
           FP8Q_OK, 1);
    if (fp8q::stub_gemm.splits != 4 || (void*)fp8q::stub_gemm.cnt != (void*)ws ||
        (void*)fp8q::stub_gemm.part != (void*)(ws + 256)) {
      fprintf(stderr, "split-K arguments: splits %d\n", fp8q::stub_gemm.splits);
      ++failures;
    }
    EXPECT(fp8q_gemm_splitk(cA, sA, FP8Q_BLOCK_1x128, 12288, cA, sA, FP8Q_BLOCK_128x128, 12288, 256, 4096, 12288, C,
                            4096, ws, ws_down - 1, nullptr),
           FP8Q_ERR_INVAL, 0);
    EXPECT(fp8q_gemm_splitk(cA, sA, FP8Q_BLOCK_1x128, 12288, cA, sA, FP8Q_BLOCK_128x128, 12288, 256, 4096, 12288, C,
                            4096, nullptr, ws_down, nullptr),
           FP8Q_ERR_INVAL, 0);
    EXPECT(fp8q_gemm_splitk(cA, sA, FP8Q_BLOCK_1x128, 12288, cA, sA, FP8Q_BLOCK_128x128, 12288, 256, 4096, 12288, C,
                            4096, ws + 8, ws_down, nullptr),
           FP8Q_ERR_ALIGN, 0);
    // not split: no workspace needed, fp8q_gemm's launch with splits = 1
    EXPECT(fp8q_gemm_splitk(cA, sA, FP8Q_BLOCK_1x128, 4096, cA, sA, FP8Q_BLOCK_128x128, 4096, 256, 12288, 4096, C,
                            12288, nullptr, 0, nullptr),
           FP8Q_OK, 1);
    if (fp8q::stub_gemm.splits != 1) {
      fprintf(stderr, "unsplit call: splits %d\n", fp8q::stub_gemm.splits);
      ++failures;
    }
    EXPECT(fp8q_gemm_splitk(cA, sA, FP8Q_BLOCK_1x128, BIG, cA, sA, FP8Q_BLOCK_128x128, BIG, BIG, BIG, 4096, C, BIG,
                            ws, ws_down, nullptr),
           FP8Q_ERR_UNSUPPORTED, 0);
  }

  // grouped
  fp8q_gemm_problem p[FP8Q_MAX_GROUP + 1];
  for (auto& q : p) q = fp8q_gemm_problem{cA, sA, 4096, cA, sA, 4096, C, 6144, 16384, 6144};
  EXPECT(fp8q_gemm_grouped(p, 3, FP8Q_BLOCK_1x128, FP8Q_BLOCK_128x128, 4096, nullptr), FP8Q_OK, 1);
  EXPECT(fp8q_gemm_grouped(p, FP8Q_MAX_GROUP + 1, FP8Q_BLOCK_1x128, FP8Q_BLOCK_128x128, 4096, nullptr),
         FP8Q_ERR_INVAL, 0);
  EXPECT(fp8q_gemm_grouped(p, 0, FP8Q_BLOCK_1x128, FP8Q_BLOCK_128x128, 4096, nullptr), FP8Q_ERR_INVAL, 0);
  p[1].M = BIG;
  p[1].ldc = BIG;
  EXPECT(fp8q_gemm_grouped(p, 2, FP8Q_BLOCK_1x128, FP8Q_BLOCK_128x128, 4096, nullptr), FP8Q_ERR_UNSUPPORTED, 0);
  p[1].M = 200000;
  p[1].ldc = 6144;
  EXPECT(fp8q_gemm_grouped(p, 2, FP8Q_BLOCK_1x128, FP8Q_BLOCK_128x128, 4096, nullptr), FP8Q_ERR_UNSUPPORTED, 0);

  // Calibrated Clipping
  fp8q_clip_config cfg{0.8, 1.24, 0.5, 0.9, 1.2, 2.0, 0.02, 0.05, 0.1};
  const float* t = fake<const float>();
  fp8q_clip_result* res = fake<fp8q_clip_result>();
  const int64_t ws = fp8q_calibrate_clip_workspace(8863490);
  EXPECT(ws > 0 && ws <= FP8Q_CLIP_SCRATCH_BYTES ? 0 : 1, 0, 0);
  EXPECT(fp8q_calibrate_clip(t, t, t, t, t, 8863490, 0.6, 1.8, &cfg, C, ws, res, nullptr), FP8Q_OK, 1);
  EXPECT(fp8q_calibrate_clip(t, t, t, t, t, 8863490, 0.6, 1.8, &cfg, C, ws - 8, res, nullptr), FP8Q_ERR_INVAL, 0);
  EXPECT(fp8q_calibrate_clip(t, t, t, t, t, BIG, 0.6, 1.8, &cfg, C, BIG, res, nullptr), FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_calibrate_clip_workspace(BIG), -1, 0);
  EXPECT(fp8q_calibrate_clip_noalloc(t, t, t, t, t, 8863490, 0.6, 1.8, &cfg, res, nullptr), FP8Q_OK, 1);
  EXPECT(fp8q_calibrate_clip_noalloc(t, t, t, t, t, BIG, 0.6, 1.8, &cfg, res, nullptr), FP8Q_ERR_UNSUPPORTED, 0);
  fp8q_clip_config bad = cfg;
  bad.step = 0.0;
  EXPECT(fp8q_calibrate_clip_noalloc(t, t, t, t, t, 100, 0.6, 1.8, &bad, res, nullptr), FP8Q_ERR_INVAL, 0);
  bad = cfg;
  bad.l_max = 1e300;
  EXPECT(fp8q_calibrate_clip_noalloc(t, t, t, t, t, 100, 0.6, 1.8, &bad, res, nullptr), FP8Q_ERR_INVAL, 0);

  // casts
  EXPECT(fp8q_cast_f32(t, 1000, 1.0f, codes, nullptr), FP8Q_OK, 1);
  EXPECT(fp8q_cast_f32(t, BIG, 1.0f, codes, nullptr), FP8Q_ERR_UNSUPPORTED, 0);
  EXPECT(fp8q_cast_f32_e5m2(t, 1000, -1.0f, codes, nullptr), FP8Q_ERR_INVAL, 0);

  printf("C-ABI host checks: %d failures\n", failures);
  return failures ? 1 : 0;
}
