// Scaled FP8 GEMM of the FP8 linear layer on gfx950:
//   C[m][n] = sum_k (S_A(m,k) A[m][k]) (S_B(n,k) B[n][k]),  A, B OCP E4M3,
// fp32 accumulation on the matrix cores, bf16 output.
//
// Tiling: a 256-thread workgroup owns a 128 x 128 tile of C; its four waves
// each own 64 x 64 as 4 x 4 MFMA tiles of 16 x 16.  The K loop steps by 128,
// which is both the depth of one v_mfma_f32_16x16x128_f8f6f4 and the length
// of one scale block, so a blockwise step is one MFMA per 16 x 16 tile into
// a zeroed partial, then one FMA per accumulator that adds S_A * S_B * P.
//
// Operand tiles (128 rows x 128 bytes of K) go global -> LDS with the
// direct-to-LDS 16-byte loads of gfx950 (no VGPR staging), double buffered.
// In LDS the 16-byte chunk c of row r is stored at chunk c ^ (r & 7), so the
// eight rows read together by a ds_read_b128 hit eight different chunks.
// The MFMA "A" operand is the B tile (rows n) and the MFMA "B" operand the A
// tile (rows m): each lane then ends with four consecutive n of one m, which
// the epilogue stores as one 8-byte bf16x4.
#include "device_common.h"
#include "internal.h"

namespace fp8q {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kBM = 128, kBN = 128, kBK = 128;
constexpr int kThreads = 256;
constexpr int kTileBytes = kBM * kBK;        // one operand tile, 16 KB
constexpr int kStageBytes = 2 * kTileBytes;  // A tile + B tile
constexpr int kGroupM = 8;                   // tile rows per group of the raster

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ v4f mfma_16x16x128(const v8i& a, const v8i& b, const v4f& c) {
  // Scale operands 0 select the unscaled E4M3 x E4M3 instruction.
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Copy one 128 x 128-byte operand tile (rows row0.., K bytes k0..) into LDS.
// Each wave moves four groups of eight rows; lane l of a group lands at byte
// 16 * l of the group's 1 KB, i.e. row l / 8, physical chunk l % 8, so it
// fetches logical chunk (l % 8) ^ (l / 8).  Rows past `rows` are clamped to
// the last row (their results are never stored).
__device__ __forceinline__ void load_tile_lds(const uint8_t* base, int64_t ld, int64_t row0, int64_t rows,
                                              int64_t k0, uint8_t* lds_tile) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int chunk = (lane & 7) ^ (lane >> 3);
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int grp = wave * 4 + g;  // 16 groups of 8 rows
    int64_t r = row0 + grp * 8 + (lane >> 3);
    r = r < rows ? r : rows - 1;
    const uint8_t* src = base + r * ld + k0 + chunk * 16;
    __builtin_amdgcn_global_load_lds((const void*)src, (lds_void*)(lds_tile + grp * 1024), 16, 0, 0);
  }
}

// 32 K-bytes of one operand row for the MFMA: logical chunks 2g and 2g+1
// of row `row` (g = lane / 16), un-swizzled.
__device__ __forceinline__ v8i read_frag(const uint8_t* lds_tile, int row) {
  const int g = (threadIdx.x & 63) >> 4;
  const int sw = row & 7;
  const uint4 lo = *reinterpret_cast<const uint4*>(lds_tile + row * 128 + (((2 * g) ^ sw) << 4));
  const uint4 hi = *reinterpret_cast<const uint4*>(lds_tile + row * 128 + (((2 * g + 1) ^ sw) << 4));
  v8i f;
  f[0] = (int)lo.x; f[1] = (int)lo.y; f[2] = (int)lo.z; f[3] = (int)lo.w;
  f[4] = (int)hi.x; f[5] = (int)hi.y; f[6] = (int)hi.z; f[7] = (int)hi.w;
  return f;
}

__device__ __forceinline__ void wait_vmem_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Tile coordinates of this workgroup.  Workgroup b runs on XCD b % 8, so
// each XCD is given a contiguous range of the raster (sharing its L2), and
// the raster walks kGroupM tile rows at a time so that consecutive tiles
// reuse A rows and B rows.
__device__ __forceinline__ void tile_coords(int64_t M, int64_t N, int& tm, int& tn) {
  const int tiles_m = (int)((M + kBM - 1) / kBM), tiles_n = (int)((N + kBN - 1) / kBN);
  const int total = tiles_m * tiles_n;
  const int b = blockIdx.x;
  const int xcd = b & 7, per = total >> 3, extra = total & 7;
  const int id = xcd * per + (xcd < extra ? xcd : extra) + (b >> 3);
  const int per_group = kGroupM * tiles_n;
  const int group = id / per_group;
  const int first_m = group * kGroupM;
  const int gsize = (tiles_m - first_m) < kGroupM ? (tiles_m - first_m) : kGroupM;
  const int in_group = id - group * per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

template <int PAIR>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * kStageBytes];

  int tm, tn;
  tile_coords(g.M, g.N, tm, tn);
  const int64_t m0 = (int64_t)tm * kBM, n0 = (int64_t)tn * kBN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;  // wave's 64 x 64 sub-tile
  const int KT = (int)(g.K / kBK);

  v4f acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  // rows of C this lane accumulates: m = m0 + wm + 16 i + lane % 16,
  // n = n0 + wn + 16 j + 4 (lane / 16) + r
  int64_t mrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + wm + i * 16 + (lane & 15);
    mrow[i] = m < g.M ? m : g.M - 1;
  }
  int64_t ncol[4][4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t n = n0 + wn + j * 16 + (lane >> 4) * 4 + r;
      ncol[j][r] = n < g.N ? n : g.N - 1;
    }

  // per-K-block scales, fetched one step ahead
  float sa[4], sb[4][4], sb0 = 0.f;
  auto fetch_scales = [&](int kt, float (&a)[4], float (&b)[4][4], float& b0) {
    if (PAIR == kPairBlock || PAIR == kPairBlockK) {
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = g.sA[(int64_t)kt * g.M + mrow[i]];
    }
    if (PAIR == kPairBlock) b0 = g.sB[(n0 / 128) * (g.K / 128) + kt];
    if (PAIR == kPairBlockK) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) b[j][r] = g.sB[(int64_t)kt * g.N + ncol[j][r]];
    }
  };

  fetch_scales(0, sa, sb, sb0);
  load_tile_lds(g.A, g.lda, m0, g.M, 0, lds);
  load_tile_lds(g.B, g.ldb, n0, g.N, 0, lds + kTileBytes);

  for (int kt = 0; kt < KT; ++kt) {
    uint8_t* cur = lds + (kt & 1) * kStageBytes;
    wait_vmem_all();
    __syncthreads();  // tile kt is in LDS for every wave; stage kt+1 is free

    float sa_n[4], sb_n[4][4], sb0_n = 0.f;
    if (kt + 1 < KT) {
      fetch_scales(kt + 1, sa_n, sb_n, sb0_n);
      uint8_t* nxt = lds + ((kt + 1) & 1) * kStageBytes;
      load_tile_lds(g.A, g.lda, m0, g.M, (int64_t)(kt + 1) * kBK, nxt);
      load_tile_lds(g.B, g.ldb, n0, g.N, (int64_t)(kt + 1) * kBK, nxt + kTileBytes);
    }

    v8i af[4], bf[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = read_frag(cur, wm + i * 16 + (lane & 15));
#pragma unroll
    for (int j = 0; j < 4; ++j) bf[j] = read_frag(cur + kTileBytes, wn + j * 16 + (lane & 15));

    if (PAIR == kPairTensor || PAIR == kPairRow) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma_16x16x128(bf[j], af[i], acc[i][j]);
    } else {
      const v4f zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const v4f p = mfma_16x16x128(bf[j], af[i], zero);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            if (PAIR == kPairBlock) {
              acc[i][j][r] = __builtin_fmaf(p[r], sa[i] * sb0, acc[i][j][r]);
            } else {
              acc[i][j][r] = __builtin_fmaf(p[r] * sa[i], sb[j][r], acc[i][j][r]);
            }
          }
        }
      }
    }

    if (kt + 1 < KT) {
#pragma unroll
      for (int i = 0; i < 4; ++i) sa[i] = sa_n[i];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) sb[j][r] = sb_n[j][r];
      sb0 = sb0_n;
    }
  }

  // epilogue: whole-K scales for tensor / row pairs, bf16 RNE, store
  float st = 1.0f;
  if (PAIR == kPairTensor) st = g.sA[0] * g.sB[0];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + wm + i * 16 + (lane & 15);
    if (m >= g.M) continue;
    const float sm = PAIR == kPairRow ? g.sA[m] : 1.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t n = n0 + wn + j * 16 + (lane >> 4) * 4;
      uint32_t h[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float v = acc[i][j][r];
        if (PAIR == kPairTensor) v = v * st;
        if (PAIR == kPairRow) v = (v * sm) * g.sB[ncol[j][r]];
        h[r] = bf16_rne(v);
      }
      uint16_t* dst = g.C + m * g.ldc + n;
      if (n + 3 < g.N) {
        *reinterpret_cast<uint2*>(dst) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (n + r < g.N) dst[r] = (uint16_t)h[r];
      }
    }
  }
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& g, int pair, hipStream_t s) {
  const int64_t tiles = ((g.M + kBM - 1) / kBM) * ((g.N + kBN - 1) / kBN);
  if (tiles <= 0 || tiles > 0x7fffffff) return hipErrorInvalidValue;
  const dim3 grid((unsigned)tiles);
  switch (pair) {
    case kPairTensor: gemm_kernel<kPairTensor><<<grid, kThreads, 0, s>>>(g); break;
    case kPairRow: gemm_kernel<kPairRow><<<grid, kThreads, 0, s>>>(g); break;
    case kPairBlock: gemm_kernel<kPairBlock><<<grid, kThreads, 0, s>>>(g); break;
    case kPairBlockK: gemm_kernel<kPairBlockK><<<grid, kThreads, 0, s>>>(g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace fp8q
