// C-ABI of libfp8q: argument validation, then kernel launches on the
// caller's stream.  Declarations and contracts are in include/fp8q.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fp8q.h"
#include "internal.h"

namespace fp8q {

// Split-K applies where the tiled kernels leave CUs without a 128 x 128
// tile (fewer than 128 tiles: a decode step's down-projection, 256 x 4096
// outputs, has 64): the largest power of two S <= 8 with at most one
// workgroup per CU (tiles x S <= 256), S dividing the K blocks and at least
// four K blocks per split.  Problems that launch_split would cut into
// sub-problems (2 GiB operand spans) are not split.
int gemm_splitk_splits(int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc) {
  const int64_t lim = (int64_t)1 << 31;
  if (M <= 0 || N <= 0 || K <= 0 || K % 128) return 1;
  if (M * lda >= lim || N * ldb >= lim || M * 2 * ldc >= lim) return 1;
  const int64_t tiles = ((M + 127) / 128) * ((N + 127) / 128), kblocks = K / 128;
  if (tiles >= 128) return 1;
  int best = 1;
  for (int sp = 2; sp <= 8; sp *= 2)
    if (tiles * sp <= 256 && kblocks % sp == 0 && kblocks / sp >= 4) best = sp;
  return best;
}

// Workspace: one 32-bit counter per tile (the counters padded to 256
// bytes), then `splits` fp32 partial tiles of 128 x 128 per tile.
int64_t gemm_splitk_workspace(int64_t M, int64_t N, int splits) {
  if (splits <= 1) return 0;
  const int64_t tiles = ((M + 127) / 128) * ((N + 127) / 128);
  return (tiles * 4 + 255) / 256 * 256 + tiles * splits * 128 * 128 * 4;
}

}  // namespace fp8q

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool valid_granularity(int g) { return g >= FP8Q_TENSOR && g <= FP8Q_BLOCK_128x128; }

// Largest size or leading dimension taken (else FP8Q_ERR_UNSUPPORTED): every
// product of two of them, doubled, stays below 2^63, so the checks and the
// launchers' offset arithmetic cannot overflow.
constexpr int64_t kMaxDim = 0x7fffffff;
bool dims_ok(int64_t a, int64_t b, int64_t c = 1, int64_t d = 1, int64_t e = 1) {
  return a <= kMaxDim && b <= kMaxDim && c <= kMaxDim && d <= kMaxDim && e <= kMaxDim;
}

constexpr unsigned kQuantFlags = FP8Q_OUT_TRANSPOSED | FP8Q_POW2_SCALE | FP8Q_E5M2;

int transposed_granularity(int g) {
  switch (g) {
    case FP8Q_ROW: return FP8Q_COL;
    case FP8Q_COL: return FP8Q_ROW;
    case FP8Q_BLOCK_1x128: return FP8Q_BLOCK_128x1;
    case FP8Q_BLOCK_128x1: return FP8Q_BLOCK_1x128;
    default: return g;
  }
}

int64_t count_for(int64_t rows, int64_t cols, int g) {
  switch (g) {
    case FP8Q_TENSOR: return 1;
    case FP8Q_ROW: return rows;
    case FP8Q_COL: return cols;
    case FP8Q_BLOCK_1x128: return rows * (cols / 128);
    case FP8Q_BLOCK_128x1: return (rows / 128) * cols;
    case FP8Q_BLOCK_128x128: return (rows / 128) * (cols / 128);
    default: return -1;
  }
}

fp8q_status from_hip(hipError_t e) { return e == hipSuccess ? FP8Q_OK : FP8Q_ERR_HIP; }

// Largest batch of Calibrated Clipping (tokens; else FP8Q_ERR_UNSUPPORTED).
constexpr int64_t kMaxClipTokens = (int64_t)1 << 52;

// Calibrated Clipping: one block per `chunk` consecutive tokens, at most
// kClipMaxBlocks (one per CU), chunks a multiple of 1024 tokens (up to 256
// threads x 4).
void clip_blocks(int64_t n, int64_t& chunk, int64_t& blocks) {
  int64_t c = (n + fp8q::kClipMaxBlocks - 1) / fp8q::kClipMaxBlocks;
  c = (c + 1023) / 1024 * 1024;
  chunk = c < 4096 ? 4096 : c;
  blocks = (n + chunk - 1) / chunk;
}

// Points lo + k step, k = 0 .. round((hi - lo) / step), when the span is a
// whole number of steps (to 1e-9 of a step).
bool grid_size(double lo, double hi, double step, int& n) {
  const double q = (hi - lo) / step;
  const double k = nearbyint(q);
  if (!(fabs(q - k) <= 1e-9) || k > 1e6) return false;
  n = (int)k + 1;
  return true;
}

// The checks of fp8q_gemm (with operand formats: FP8Q_A_E5M2 / FP8Q_B_E5M2
// bits, only for the two blockwise pairs), then the kernel arguments.
fp8q_status gemm_args(const uint8_t* A, const float* sA, fp8q_granularity gA, int64_t lda, const uint8_t* B,
                      const float* sB, fp8q_granularity gB, int64_t ldb, int64_t M, int64_t N, int64_t K,
                      unsigned formats, void* C, int64_t ldc, fp8q::GemmArgs& g, int& pair) {
  if (!A || !sA || !B || !sB || !C) return FP8Q_ERR_INVAL;
  if (formats & ~(unsigned)(FP8Q_A_E5M2 | FP8Q_B_E5M2)) return FP8Q_ERR_INVAL;
  if (M <= 0 || N <= 0 || K <= 0 || !valid_granularity(gA) || !valid_granularity(gB)) return FP8Q_ERR_INVAL;
  if (lda < K || ldb < K || ldc < N) return FP8Q_ERR_INVAL;
  if (!dims_ok(M, N, lda, ldb, ldc)) return FP8Q_ERR_UNSUPPORTED;
  if (gA == FP8Q_TENSOR && gB == FP8Q_TENSOR)
    pair = fp8q::kPairTensor;
  else if (gA == FP8Q_ROW && gB == FP8Q_ROW)
    pair = fp8q::kPairRow;
  else if (gA == FP8Q_BLOCK_1x128 && gB == FP8Q_BLOCK_128x128)
    pair = fp8q::kPairBlock;
  else if (gA == FP8Q_BLOCK_1x128 && gB == FP8Q_BLOCK_1x128)
    pair = fp8q::kPairBlockK;
  else
    return FP8Q_ERR_UNSUPPORTED;
  if (formats && pair != fp8q::kPairBlock && pair != fp8q::kPairBlockK) return FP8Q_ERR_UNSUPPORTED;
  if (K % 128 || (gB == FP8Q_BLOCK_128x128 && N % 128)) return FP8Q_ERR_UNSUPPORTED;
  if (((M + 127) / 128) * ((N + 127) / 128) > 0x7fffffff) return FP8Q_ERR_UNSUPPORTED;
  if (!aligned(A, 16) || !aligned(B, 16) || lda % 16 || ldb % 16 || !aligned(C, 8) || ldc % 4 ||
      !aligned(sA, 4) || !aligned(sB, 4))
    return FP8Q_ERR_ALIGN;
  g.A = A;
  g.B = B;
  g.sA = sA;
  g.sB = sB;
  g.C = static_cast<uint16_t*>(C);
  g.M = M;
  g.N = N;
  g.K = K;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.sa_ld = M;
  g.sb_ld = N;
  g.sa_count = count_for(M, K, gA);
  g.sb_count = count_for(N, K, gB);
  g.c_aligned16 = aligned(C, 16) && ldc % 8 == 0;
  g.Cq = nullptr;
  g.Cs = nullptr;
  g.ldq = 0;
  g.cs_ld = 0;
  return FP8Q_OK;
}

fp8q_status gemm_checked(const uint8_t* A, const float* sA, fp8q_granularity gA, int64_t lda, const uint8_t* B,
                         const float* sB, fp8q_granularity gB, int64_t ldb, int64_t M, int64_t N, int64_t K,
                         unsigned formats, void* C, int64_t ldc, struct ihipStream_t* stream) {
  fp8q::GemmArgs g;
  int pair = 0;
  const fp8q_status st = gemm_args(A, sA, gA, lda, B, sB, gB, ldb, M, N, K, formats, C, ldc, g, pair);
  if (st != FP8Q_OK) return st;
  return from_hip(fp8q::launch_gemm(g, pair, (int)formats, reinterpret_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" {

int64_t fp8q_scales_count(int64_t rows, int64_t cols, fp8q_granularity g, unsigned flags) {
  if (rows <= 0 || cols <= 0 || !valid_granularity(g) || (flags & ~kQuantFlags) || !dims_ok(rows, cols))
    return -1;
  const bool t = (flags & FP8Q_OUT_TRANSPOSED) != 0;
  const int64_t orows = t ? cols : rows, ocols = t ? rows : cols;
  return count_for(orows, ocols, t ? transposed_granularity(g) : g);
}

fp8q_status fp8q_quantize(const void* x, int64_t rows, int64_t cols, int64_t ldx, fp8q_granularity g,
                          unsigned flags, uint8_t* codes, int64_t ldc, float* scales,
                          struct ihipStream_t* stream) {
  if (!x || !codes || !scales) return FP8Q_ERR_INVAL;
  if (rows <= 0 || cols <= 0 || !valid_granularity(g) || (flags & ~kQuantFlags)) return FP8Q_ERR_INVAL;
  const bool t = (flags & FP8Q_OUT_TRANSPOSED) != 0;
  if (ldx < cols || ldc < (t ? rows : cols)) return FP8Q_ERR_INVAL;
  if (!dims_ok(rows, cols, ldx, ldc)) return FP8Q_ERR_UNSUPPORTED;
  const bool splits_cols = g == FP8Q_BLOCK_1x128 || g == FP8Q_BLOCK_128x128;
  const bool splits_rows = g == FP8Q_BLOCK_128x1 || g == FP8Q_BLOCK_128x128;
  if (cols % 16 || (t && rows % 16)) return FP8Q_ERR_UNSUPPORTED;
  if ((splits_cols && cols % 128) || (splits_rows && rows % 128)) return FP8Q_ERR_UNSUPPORTED;
  if (rows > (int64_t)65535 * 128) return FP8Q_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scales, 4) || ldx % 8 || ldc % 16)
    return FP8Q_ERR_ALIGN;
  fp8q::QuantArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.rows = rows;
  a.cols = cols;
  a.ldx = ldx;
  a.codes = codes;
  a.ldc = ldc;
  a.scales = scales;
  a.pow2 = (flags & FP8Q_POW2_SCALE) != 0;
  a.e5m2 = (flags & FP8Q_E5M2) != 0;
  const int64_t n = fp8q_scales_count(rows, cols, g, flags);
  return from_hip(fp8q::launch_quantize(a, g, t, n, reinterpret_cast<hipStream_t>(stream)));
}

fp8q_status fp8q_quantize_dual(const void* x, int64_t rows, int64_t cols, int64_t ldx, unsigned flags,
                               uint8_t* codes_r, int64_t ldc_r, float* scales_r, uint8_t* codes_t, int64_t ldc_t,
                               float* scales_t, struct ihipStream_t* stream) {
  if (!x || !codes_r || !scales_r || !codes_t || !scales_t) return FP8Q_ERR_INVAL;
  if (flags & ~(unsigned)(FP8Q_POW2_SCALE | FP8Q_E5M2)) return FP8Q_ERR_INVAL;
  if (rows <= 0 || cols <= 0 || ldx < cols || ldc_r < cols || ldc_t < rows) return FP8Q_ERR_INVAL;
  if (!dims_ok(rows, cols, ldx, ldc_r, ldc_t)) return FP8Q_ERR_UNSUPPORTED;
  if (rows % 128 || cols % 128) return FP8Q_ERR_UNSUPPORTED;
  if (rows > (int64_t)65535 * 128) return FP8Q_ERR_UNSUPPORTED;  // grid.y limit
  if (!aligned(x, 16) || !aligned(codes_r, 16) || !aligned(codes_t, 16) || !aligned(scales_r, 4) ||
      !aligned(scales_t, 4) || ldx % 8 || ldc_r % 16 || ldc_t % 16)
    return FP8Q_ERR_ALIGN;
  fp8q::DualArgs d;
  d.a.x = static_cast<const uint16_t*>(x);
  d.a.rows = rows;
  d.a.cols = cols;
  d.a.ldx = ldx;
  d.a.codes = codes_r;
  d.a.ldc = ldc_r;
  d.a.scales = scales_r;
  d.a.pow2 = (flags & FP8Q_POW2_SCALE) != 0;
  d.a.e5m2 = (flags & FP8Q_E5M2) != 0;
  d.codes_t = codes_t;
  d.ldc_t = ldc_t;
  d.scales_t = scales_t;
  return from_hip(fp8q::launch_quantize_dual(d, reinterpret_cast<hipStream_t>(stream)));
}

fp8q_status fp8q_gemm(const uint8_t* A, const float* sA, fp8q_granularity gA, int64_t lda, const uint8_t* B,
                      const float* sB, fp8q_granularity gB, int64_t ldb, int64_t M, int64_t N, int64_t K,
                      void* C, int64_t ldc, struct ihipStream_t* stream) {
  return gemm_checked(A, sA, gA, lda, B, sB, gB, ldb, M, N, K, 0u, C, ldc, stream);
}

int64_t fp8q_gemm_splitk_workspace(int64_t M, int64_t N, int64_t K) {
  if (M <= 0 || N <= 0 || K <= 0 || M > kMaxDim || N > kMaxDim || K > kMaxDim) return -1;
  return fp8q::gemm_splitk_workspace(M, N, fp8q::gemm_splitk_splits(M, N, K, K, K, N));
}

fp8q_status fp8q_gemm_splitk(const uint8_t* A, const float* sA, fp8q_granularity gA, int64_t lda, const uint8_t* B,
                             const float* sB, fp8q_granularity gB, int64_t ldb, int64_t M, int64_t N, int64_t K,
                             void* C, int64_t ldc, void* workspace, int64_t workspace_bytes,
                             struct ihipStream_t* stream) {
  fp8q::GemmArgs g;
  int pair = 0;
  const fp8q_status st = gemm_args(A, sA, gA, lda, B, sB, gB, ldb, M, N, K, 0u, C, ldc, g, pair);
  if (st != FP8Q_OK) return st;
  g.splits = fp8q::gemm_splitk_splits(M, N, K, lda, ldb, ldc);
  if (g.splits > 1) {
    const int64_t need = fp8q::gemm_splitk_workspace(M, N, g.splits);
    if (!workspace || workspace_bytes < need) return FP8Q_ERR_INVAL;
    if (!aligned(workspace, 16)) return FP8Q_ERR_ALIGN;
    const int64_t tiles = ((M + 127) / 128) * ((N + 127) / 128);
    g.cnt = static_cast<uint32_t*>(workspace);
    g.part = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + (tiles * 4 + 255) / 256 * 256);
  }
  return from_hip(fp8q::launch_gemm_splitk(g, pair, reinterpret_cast<hipStream_t>(stream)));
}

fp8q_status fp8q_gemm_formats(const uint8_t* A, const float* sA, fp8q_granularity gA, int64_t lda,
                              const uint8_t* B, const float* sB, fp8q_granularity gB, int64_t ldb, int64_t M,
                              int64_t N, int64_t K, unsigned formats, void* C, int64_t ldc,
                              struct ihipStream_t* stream) {
  return gemm_checked(A, sA, gA, lda, B, sB, gB, ldb, M, N, K, formats, C, ldc, stream);
}

fp8q_status fp8q_gemm_grouped(const fp8q_gemm_problem* problems, int count, fp8q_granularity gA,
                              fp8q_granularity gB, int64_t K, struct ihipStream_t* stream) {
  if (!problems || count < 1 || count > FP8Q_MAX_GROUP) return FP8Q_ERR_INVAL;
  static_assert(FP8Q_MAX_GROUP == fp8q::kMaxGroup, "group limits agree");
  fp8q::GemmGroup gs;
  int pair = 0;
  const int64_t lim = (int64_t)1 << 31;
  for (int i = 0; i < count; ++i) {
    const fp8q_gemm_problem& p = problems[i];
    const fp8q_status st =
        gemm_args(p.A, p.sA, gA, p.lda, p.B, p.sB, gB, p.ldb, p.M, p.N, K, 0u, p.C, p.ldc, gs.prob[i], pair);
    if (st != FP8Q_OK) return st;
    if (pair == fp8q::kPairBlockK) return FP8Q_ERR_UNSUPPORTED;
    // the kernel's 32-bit operand offsets (fp8q_gemm splits such a problem)
    if (p.M * p.lda >= lim || p.N * p.ldb >= lim || p.M * 2 * p.ldc >= lim) return FP8Q_ERR_UNSUPPORTED;
  }
  gs.count = count;
  return from_hip(fp8q::launch_gemm_grouped(gs, pair, reinterpret_cast<hipStream_t>(stream)));
}

fp8q_status fp8q_gemm_pow2(const uint8_t* A, const float* sA, fp8q_granularity gA, int64_t lda, const uint8_t* B,
                           const float* sB, fp8q_granularity gB, int64_t ldb, int64_t M, int64_t N, int64_t K,
                           void* C, int64_t ldc, struct ihipStream_t* stream) {
  if (!A || !sA || !B || !sB || !C) return FP8Q_ERR_INVAL;
  if (M <= 0 || N <= 0 || K <= 0 || !valid_granularity(gA) || !valid_granularity(gB)) return FP8Q_ERR_INVAL;
  if (lda < K || ldb < K || ldc < N) return FP8Q_ERR_INVAL;
  if (!dims_ok(M, N, lda, ldb, ldc)) return FP8Q_ERR_UNSUPPORTED;
  if (gA != FP8Q_BLOCK_1x128 || gB != FP8Q_BLOCK_128x128) return FP8Q_ERR_UNSUPPORTED;
  if (K % 128 || N % 128) return FP8Q_ERR_UNSUPPORTED;
  if (((M + 127) / 128) * (N / 128) > 0x7fffffff) return FP8Q_ERR_UNSUPPORTED;
  if (!aligned(A, 16) || !aligned(B, 16) || lda % 16 || ldb % 16 || !aligned(C, 8) || ldc % 4 ||
      !aligned(sA, 4) || !aligned(sB, 4))
    return FP8Q_ERR_ALIGN;
  fp8q::GemmArgs g;
  g.A = A;
  g.B = B;
  g.sA = sA;
  g.sB = sB;
  g.C = static_cast<uint16_t*>(C);
  g.M = M;
  g.N = N;
  g.K = K;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.sa_ld = M;
  g.sb_ld = N;
  g.sa_count = count_for(M, K, gA);
  g.sb_count = count_for(N, K, gB);
  g.c_aligned16 = aligned(C, 16) && ldc % 8 == 0;
  g.Cq = nullptr;
  g.Cs = nullptr;
  g.ldq = 0;
  g.cs_ld = 0;
  return from_hip(fp8q::launch_gemm(g, fp8q::kPairBlockE8, 0, reinterpret_cast<hipStream_t>(stream)));
}

fp8q_status fp8q_gemm_quantized(const uint8_t* A, const float* sA, fp8q_granularity gA, int64_t lda,
                                const uint8_t* B, const float* sB, fp8q_granularity gB, int64_t ldb, int64_t M,
                                int64_t N, int64_t K, uint8_t* codes, int64_t ldq, float* scales,
                                struct ihipStream_t* stream) {
  if (!A || !sA || !B || !sB || !codes || !scales) return FP8Q_ERR_INVAL;
  if (M <= 0 || N <= 0 || K <= 0 || !valid_granularity(gA) || !valid_granularity(gB)) return FP8Q_ERR_INVAL;
  if (lda < K || ldb < K || ldq < N) return FP8Q_ERR_INVAL;
  if (!dims_ok(M, N, lda, ldb, ldq)) return FP8Q_ERR_UNSUPPORTED;
  if (gA != FP8Q_BLOCK_1x128 || gB != FP8Q_BLOCK_128x128) return FP8Q_ERR_UNSUPPORTED;
  if (K % 128 || N % 128) return FP8Q_ERR_UNSUPPORTED;
  if (((M + 127) / 128) * (N / 128) > 0x7fffffff) return FP8Q_ERR_UNSUPPORTED;
  if (!aligned(A, 16) || !aligned(B, 16) || lda % 16 || ldb % 16 || !aligned(codes, 16) || ldq % 16 ||
      !aligned(sA, 4) || !aligned(sB, 4) || !aligned(scales, 4))
    return FP8Q_ERR_ALIGN;
  fp8q::GemmArgs g;
  g.A = A;
  g.B = B;
  g.sA = sA;
  g.sB = sB;
  g.C = nullptr;
  g.M = M;
  g.N = N;
  g.K = K;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = N;
  g.sa_ld = M;
  g.sb_ld = N;
  g.sa_count = count_for(M, K, gA);
  g.sb_count = count_for(N, K, gB);
  g.c_aligned16 = 0;
  g.Cq = codes;
  g.Cs = scales;
  g.ldq = ldq;
  g.cs_ld = M;
  return from_hip(fp8q::launch_gemm_quantized(g, fp8q::kPairBlock, reinterpret_cast<hipStream_t>(stream)));
}

int64_t fp8q_calibrate_clip_workspace(int64_t n) {
  if (n <= 0 || n > kMaxClipTokens) return -1;
  int64_t chunk, blocks;
  clip_blocks(n, chunk, blocks);
  return blocks * fp8q::clip_slots(fp8q::kClipMaxL, fp8q::kClipMaxH) * (int64_t)sizeof(double);
}

namespace {

// The checks shared by both Calibrated Clipping entry points (all but the
// workspace's), then the kernel arguments without the partials' address.
fp8q_status clip_args(const float* adv, const float* w_tis, const float* pi_sampler, const float* r_bf16,
                      const float* r_fp8, int64_t n, double l_old, double h_old, const fp8q_clip_config* config,
                      fp8q_clip_result* result, fp8q::ClipArgs& p) {
  if (!adv || !w_tis || !pi_sampler || !r_bf16 || !r_fp8 || !config || !result) return FP8Q_ERR_INVAL;
  if (n <= 0) return FP8Q_ERR_INVAL;
  if (n > kMaxClipTokens) return FP8Q_ERR_UNSUPPORTED;
  const fp8q_clip_config c = *config;
  if (!(c.step > 0.0) || !(c.l_max >= c.l_min) || !(c.h_max >= c.h_min)) return FP8Q_ERR_INVAL;
  int nl, nh;
  if (!grid_size(c.l_min, c.l_max, c.step, nl) || !grid_size(c.h_min, c.h_max, c.step, nh)) return FP8Q_ERR_INVAL;
  if (nl > fp8q::kClipMaxL || nh > fp8q::kClipMaxH) return FP8Q_ERR_UNSUPPORTED;
  if (!aligned(adv, 16) || !aligned(w_tis, 16) || !aligned(pi_sampler, 16) || !aligned(r_bf16, 16) ||
      !aligned(r_fp8, 16) || !aligned(result, 8))
    return FP8Q_ERR_ALIGN;
  p.adv = adv;
  p.w = w_tis;
  p.pi = pi_sampler;
  p.rb = r_bf16;
  p.rf = r_fp8;
  p.n = n;
  int64_t blocks;
  clip_blocks(n, p.chunk, blocks);
  p.blocks = (int)blocks;
  p.nl = nl;
  p.nh = nh;
  p.c_low_ref = c.c_low_ref;
  p.c_high_ref = c.c_high_ref;
  p.l_min = c.l_min;
  p.h_min = c.h_min;
  p.step = c.step;
  p.inv_step = 1.0 / c.step;
  p.delta_l = c.delta_l;
  p.delta_h = c.delta_h;
  p.l_old = l_old;
  p.h_old = h_old;
  p.partials = nullptr;
  p.result = result;
  return FP8Q_OK;
}

}  // namespace

fp8q_status fp8q_calibrate_clip(const float* adv, const float* w_tis, const float* pi_sampler, const float* r_bf16,
                                const float* r_fp8, int64_t n, double l_old, double h_old,
                                const fp8q_clip_config* config, void* workspace, int64_t workspace_bytes,
                                fp8q_clip_result* result, struct ihipStream_t* stream) {
  fp8q::ClipArgs p;
  const fp8q_status st = clip_args(adv, w_tis, pi_sampler, r_bf16, r_fp8, n, l_old, h_old, config, result, p);
  if (st != FP8Q_OK) return st;
  if (!workspace || workspace_bytes < fp8q_calibrate_clip_workspace(n)) return FP8Q_ERR_INVAL;
  if (!aligned(workspace, 8)) return FP8Q_ERR_ALIGN;
  p.partials = static_cast<double*>(workspace);
  return from_hip(fp8q::launch_calibrate_clip(p, reinterpret_cast<hipStream_t>(stream)));
}

fp8q_status fp8q_calibrate_clip_noalloc(const float* adv, const float* w_tis, const float* pi_sampler,
                                        const float* r_bf16, const float* r_fp8, int64_t n, double l_old,
                                        double h_old, const fp8q_clip_config* config, fp8q_clip_result* result,
                                        struct ihipStream_t* stream) {
  fp8q::ClipArgs p;
  const fp8q_status st = clip_args(adv, w_tis, pi_sampler, r_bf16, r_fp8, n, l_old, h_old, config, result, p);
  if (st != FP8Q_OK) return st;
  // the partials of any batch fit (at most kClipMaxBlocks blocks); checked
  // all the same, before anything is enqueued
  if (fp8q_calibrate_clip_workspace(n) > fp8q::kClipScratchBytes) return FP8Q_ERR_UNSUPPORTED;
  const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  double* partials = nullptr;
  if (fp8q::clip_scratch(s, &partials) != hipSuccess) return FP8Q_ERR_HIP;
  p.partials = partials;
  return from_hip(fp8q::launch_calibrate_clip(p, s));
}

fp8q_status fp8q_cast_f32(const float* x, int64_t n, float scale, uint8_t* codes, struct ihipStream_t* stream) {
  if (!x || !codes || n <= 0 || !(scale > 0.0f)) return FP8Q_ERR_INVAL;
  if (n > ((int64_t)1 << 62)) return FP8Q_ERR_UNSUPPORTED;
  if (!aligned(x, 4)) return FP8Q_ERR_ALIGN;
  return from_hip(fp8q::launch_cast_f32(x, n, scale, false, codes, reinterpret_cast<hipStream_t>(stream)));
}

fp8q_status fp8q_cast_f32_e5m2(const float* x, int64_t n, float scale, uint8_t* codes,
                               struct ihipStream_t* stream) {
  if (!x || !codes || n <= 0 || !(scale > 0.0f)) return FP8Q_ERR_INVAL;
  if (n > ((int64_t)1 << 62)) return FP8Q_ERR_UNSUPPORTED;
  if (!aligned(x, 4)) return FP8Q_ERR_ALIGN;
  return from_hip(fp8q::launch_cast_f32(x, n, scale, true, codes, reinterpret_cast<hipStream_t>(stream)));
}

const char* fp8q_status_string(fp8q_status s) {
  switch (s) {
    case FP8Q_OK: return "FP8Q_OK";
    case FP8Q_ERR_INVAL: return "FP8Q_ERR_INVAL: invalid argument";
    case FP8Q_ERR_UNSUPPORTED: return "FP8Q_ERR_UNSUPPORTED: unsupported shape or granularity";
    case FP8Q_ERR_ALIGN: return "FP8Q_ERR_ALIGN: misaligned pointer or leading dimension";
    case FP8Q_ERR_HIP: return "FP8Q_ERR_HIP: HIP launch failed";
    default: return "unknown fp8q status";
  }
}

}  // extern "C"
