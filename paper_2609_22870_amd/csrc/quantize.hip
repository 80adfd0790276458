// FP8 scaled quantization (Eq. 3 of the paper, Sec. 2.2) on gfx950.
//
// Every kernel works on 128 x 128 tiles of the bf16 input with 256 threads.
// Thread t holds rows 8*(t/16) .. 8*(t/16)+7 of the tile and the eight
// columns 8*(t%16) .. 8*(t%16)+7, read as one 16-byte load per row, so each
// load instruction of a wave covers four 256-byte row segments.  The sixteen
// lanes of a DPP row then hold one full 128-element tile row, which makes the
// 1x128 amax a four-step DPP reduction; 128x1 and 128x128 amaxes add a
// cross-row shuffle and one LDS exchange between the four waves.
//
// Granularities whose units span several tiles (tensor, column, and row with
// transposed output) run in three kernels: an amax pass in which every
// workgroup writes its own partial maxima (no atomics: thousands of them on
// one address serialize), a small pass that reduces the partials of each
// unit to its S, and the cast pass.  The partials live in the caller's code
// array, which the cast overwrites afterwards (in `scales` when each unit
// has a single partial).
#include "device_common.h"
#include "internal.h"

namespace fp8q {

namespace quant_detail {

constexpr int kTile = 128;
constexpr int kWideRows = 32, kWideCols = 512;
constexpr int kThreads = 256;

enum Kind { kBlock1x128, kBlock128x1, kBlock128x128, kPreTensor, kPreRow, kPreCol };

struct Tile {
  float v[8][8];  // [row i][column j] of this thread's 8 x 8 patch
};

// Rows row0 .. row0+7, columns c .. c+7 of x (zeros outside).
__device__ __forceinline__ void load_patch(const QuantArgs& a, int64_t row0, int64_t c, Tile& t) {
  const bool col_ok = c < a.cols;
  uint4 w[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int64_t r = row0 + i;
    w[i] = make_uint4(0u, 0u, 0u, 0u);
    if (col_ok && r < a.rows) w[i] = *reinterpret_cast<const uint4*>(a.x + r * a.ldx + c);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    t.v[i][0] = bf16_lo(w[i].x);
    t.v[i][1] = bf16_hi(w[i].x);
    t.v[i][2] = bf16_lo(w[i].y);
    t.v[i][3] = bf16_hi(w[i].y);
    t.v[i][4] = bf16_lo(w[i].z);
    t.v[i][5] = bf16_hi(w[i].z);
    t.v[i][6] = bf16_lo(w[i].w);
    t.v[i][7] = bf16_hi(w[i].w);
  }
}

__device__ __forceinline__ float row_partial_max(const Tile& t, int i) {
  float m = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) m = fmaxf(m, fabsf(t.v[i][j]));
  return m;
}

__device__ __forceinline__ float col_partial_max(const Tile& t, int j) {
  float m = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) m = fmaxf(m, fabsf(t.v[i][j]));
  return m;
}

// Column maxima over the whole 128-row tile: eight per thread (its columns).
__device__ __forceinline__ void tile_col_max(const Tile& t, float* lds_cols /*[4][128]*/, float out[8]) {
  const int cc = threadIdx.x & 15, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    float m = across_rows_max(col_partial_max(t, j));
    if (lane < 16) lds_cols[wave * kTile + cc * 8 + j] = m;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int col = cc * 8 + j;
    out[j] = fmaxf(fmaxf(lds_cols[col], lds_cols[kTile + col]),
                   fmaxf(lds_cols[2 * kTile + col], lds_cols[3 * kTile + col]));
  }
}

__device__ __forceinline__ float tile_max(const Tile& t, float* lds4) {
  float m = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) m = fmaxf(m, row_partial_max(t, i));
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) lds4[threadIdx.x >> 6] = m;
  __syncthreads();
  return fmaxf(fmaxf(lds4[0], lds4[1]), fmaxf(lds4[2], lds4[3]));
}

// The quotient for units of any scale, out of line: only waves holding a
// unit with S < 2^-90 call it, and keeping its IEEE divisions out of the
// kernel body keeps the common path's register use low.
__device__ __noinline__ float slow_quotient(float x, float s, float r) {
  return quotient(x, UnitScale{s, r, s >= 0x1p-90f});
}

// Which of a thread's 8 x 8 elements share a unit: its rows, its columns, or
// all of them.
enum UnitMap { kUnitRow, kUnitCol, kUnitOne };

// Codes of a thread's 8 x 8 patch (E4M3, or E5M2 when E5), two bytes per
// conversion: byte j of
// packed[i][j / 4] is element (i, j), with the unit scales su (S) and ru
// (1/S) indexed by row, by column, or [0].  The reciprocal-based quotient
// holds for S >= 2^-90 (see quotient()); waves whose units all satisfy it
// take the branch-free path.
template <int MAP, bool E5>
__device__ __forceinline__ void encode_patch(const Tile& t, const float (&su)[8], const float (&ru)[8],
                                             uint32_t (&packed)[8][2]) {
  bool fast = true;
#pragma unroll
  for (int i = 0; i < 8; ++i) fast = fast && su[i] >= 0x1p-90f;
  auto encode_all = [&](auto qf) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float q[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int j = h * 4 + jj;
          const int u = MAP == kUnitRow ? i : (MAP == kUnitCol ? j : 0);
          q[jj] = qf(t.v[i][j], su[u], ru[u]);
        }
        uint32_t w = fp8_pack2<E5, false>(q[0], q[1], 0u);
        packed[i][h] = fp8_pack2<E5, true>(q[2], q[3], w);
      }
    }
  };
  if (__all(fast))
    encode_all([](float x, float s_, float r_) { return fast_quotient(x, s_, r_); });
  else
    encode_all([](float x, float s_, float r_) { return slow_quotient(x, s_, r_); });
}

// The per-unit constants of a unit whose S is known (the cast pass of the
// multi-tile granularities): the same values unit_scale gives for its amax.
__device__ __forceinline__ UnitScale unit_of_scale(float s) { return UnitScale{s, 1.0f / s, s >= 0x1p-90f}; }

// Per-unit scales when a thread's eight rows are eight units shared by the
// 16 lanes of its DPP row: lane cc of the row group holds the amax of row
// cc % 8, computes that unit's S and 1/S (two IEEE divisions), and the
// group exchanges them by lane shuffles.
template <bool E5, bool KNOWN = false>
__device__ __forceinline__ void share_row_units(float amax, bool pow2, UnitScale& mine, float (&su)[8],
                                                float (&ru)[8]) {
  const int lane = threadIdx.x & 63;
  mine = KNOWN ? unit_of_scale(amax) : unit_scale_fmt<E5>(amax, pow2);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    su[i] = __shfl(mine.s, (lane & 48) | i, 64);
    ru[i] = __shfl(mine.r, (lane & 48) | i, 64);
  }
}

// Per-unit scales when a thread's eight columns are eight units: thread
// (rg < 8, cc) holds the amax of column 8 cc + rg, computes its S and 1/S,
// and the block exchanges them through LDS (the upper half of lds_red, after
// every read of its lower half).
template <bool E5, bool KNOWN = false>
__device__ __forceinline__ void share_col_units(float amax, bool pow2, float* lds_red, UnitScale& mine,
                                                float (&su)[8], float (&ru)[8]) {
  const int cc = threadIdx.x & 15, rg = threadIdx.x >> 4;
  mine = KNOWN ? unit_of_scale(amax) : unit_scale_fmt<E5>(amax, pow2);
  float2* lds_su = reinterpret_cast<float2*>(lds_red + 2 * kTile);
  __syncthreads();
  if (rg < 8) lds_su[cc * 8 + rg] = make_float2(mine.s, mine.r);
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float2 v = lds_su[cc * 8 + j];
    su[j] = v.x;
    ru[j] = v.y;
  }
}

// The 1x128 amax of the row this lane computes (row cc % 8 of its eight):
// each tile row is one 128-column unit spread over a 16-lane DPP row.
__device__ __forceinline__ float block_row_amax(const Tile& t) {
  const int cc = threadIdx.x & 15;
  float am[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) am[i] = row16_max(row_partial_max(t, i));
  float amax = am[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) amax = (cc & 7) == i ? am[i] : amax;
  return amax;
}

// Codes of the thread's 8 x 8 patch in the input's layout: rows row0 ..
// row0+7, columns c .. c+7.
__device__ __forceinline__ void store_patch(const uint32_t (&packed)[8][2], uint8_t* codes, int64_t ldc, int64_t rows,
                                            int64_t cols, int64_t row0, int64_t c) {
  if (c < cols) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t r = row0 + i;
      if (r < rows) *reinterpret_cast<uint2*>(codes + r * ldc + c) = make_uint2(packed[i][0], packed[i][1]);
    }
  }
}

// Codes of a 128 x 128 tile at (r0, c0) written transposed, codes[c][r],
// through LDS: LDS row = tile column (128 bytes = 16 chunks of 8 rows);
// chunk rg of LDS row 8*cc+j is stored at chunk rg ^ cc, which spreads the
// 16 lanes of a DPP row over all 32 banks.  Each output row then goes out as
// 16-byte pieces.
__device__ __forceinline__ void store_patch_transposed(const uint32_t (&packed)[8][2], uint64_t* lds_t,
                                                       uint8_t* codes, int64_t ldc, int64_t rows, int64_t cols,
                                                       int64_t r0, int64_t c0) {
  const int cc = threadIdx.x & 15, rg = threadIdx.x >> 4;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) lo |= ((packed[i][j >> 2] >> (8 * (j & 3))) & 0xffu) << (8 * i);
#pragma unroll
    for (int i = 4; i < 8; ++i) hi |= ((packed[i][j >> 2] >> (8 * (j & 3))) & 0xffu) << (8 * (i - 4));
    const int lrow = cc * 8 + j;
    lds_t[lrow * 16 + (rg ^ cc)] = (uint64_t)lo | ((uint64_t)hi << 32);
  }
  __syncthreads();
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int orow = p * 32 + (threadIdx.x >> 3);  // tile column = output row
    const int qd = threadIdx.x & 7;                // 16-byte chunk of the output row
    const int sw = orow >> 3;
    const uint64_t a0 = lds_t[orow * 16 + ((2 * qd) ^ sw)];
    const uint64_t a1 = lds_t[orow * 16 + ((2 * qd + 1) ^ sw)];
    const int64_t oc = c0 + orow;
    const int64_t orr = r0 + qd * 16;
    if (oc < cols && orr < rows)
      *reinterpret_cast<uint4*>(codes + oc * ldc + orr) =
          make_uint4((uint32_t)a0, (uint32_t)(a0 >> 32), (uint32_t)a1, (uint32_t)(a1 >> 32));
  }
}

template <int K, bool TRANS, bool E5>
__global__ __launch_bounds__(kThreads) void quant_tile_kernel(QuantArgs a) {
  __shared__ float lds_red[4 * kTile];
  __shared__ uint64_t lds_t[TRANS ? kTile * kTile / 8 : 1];

  // Row units without transposition use wide tiles of 32 x 512: wave w
  // takes rows 8 w .. 8 w + 7 and each load instruction reads one row's
  // 1 KB (four 128-column blocks, one per 16-lane group).  The others use
  // 128 x 128 tiles: thread (rg, cc) takes rows 8 rg .. 8 rg + 7.  Either
  // way a thread holds 8 rows x 8 columns, and the 16 lanes of a DPP row
  // share the thread's rows and cover 128 consecutive columns.
  constexpr bool kWide = !TRANS && (K == kBlock1x128 || K == kPreRow || K == kPreTensor);
  const int cc = threadIdx.x & 15, rg = threadIdx.x >> 4;
  const int64_t tr = blockIdx.y, tc = blockIdx.x, tiles_r = gridDim.y, tiles_c = gridDim.x;
  const int64_t r0 = tr * (kWide ? kWideRows : kTile);
  const int64_t c0 = tc * (kWide ? kWideCols : kTile);
  const int64_t row0 = kWide ? r0 + (threadIdx.x >> 6) * 8 : r0 + rg * 8;  // first of the thread's rows
  const int64_t c = kWide ? c0 + ((threadIdx.x >> 4) & 3) * 128 + cc * 8 : c0 + cc * 8;

  Tile t;
  load_patch(a, row0, c, t);

  // Per-unit scales.  A thread's elements belong to eight units (its rows for
  // 1x128 and ROW, its columns for 128x1 and COL) or to one (128x128,
  // TENSOR).  In the eight-unit case each unit's S and 1/S (two IEEE
  // divisions) are computed once, by one of the threads that share the unit,
  // and handed to the others: for rows, lane cc of a 16-lane row group
  // computes row cc % 8 and the group exchanges by lane shuffles; for
  // columns, thread (rg, cc) with rg < 8 computes column 8 cc + rg and the
  // block exchanges through LDS.
  constexpr bool by_row = K == kBlock1x128 || K == kPreRow;
  constexpr bool by_col = K == kBlock128x1 || K == kPreCol;
  UnitScale mine;  // the unit this thread computes (eight-unit case)
  float su[8], ru[8];
  if (by_row) {
    if (K == kBlock1x128) {
      const float amax = block_row_amax(t);
      share_row_units<E5>(amax, a.pow2 != 0, mine, su, ru);
    } else {
      // ROW with transposed output: S of each row, from the reduce pass
      const int64_t r = row0 + (cc & 7);
      share_row_units<E5, true>(r < a.rows ? a.scales[r] : 1.0f, false, mine, su, ru);
    }
  } else if (by_col) {
    float amax;
    if (K == kBlock128x1) {
      float m[8];
      tile_col_max(t, lds_red, m);
      amax = m[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) amax = (rg & 7) == j ? m[j] : amax;
      share_col_units<E5>(amax, a.pow2 != 0, lds_red, mine, su, ru);
    } else {
      // COL: S of each column, from the reduce pass
      const int64_t cj = c0 + cc * 8 + (rg & 7);
      share_col_units<E5, true>(cj < a.cols ? a.scales[cj] : 1.0f, false, lds_red, mine, su, ru);
    }
  } else {
    // 128x128: the tile's amax; TENSOR: S from the reduce pass
    mine = K == kBlock128x128 ? unit_scale_fmt<E5>(tile_max(t, lds_red), a.pow2 != 0) : unit_of_scale(a.scales[0]);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      su[i] = mine.s;
      ru[i] = mine.r;
    }
  }

  uint32_t packed[8][2];
  encode_patch<by_row ? kUnitRow : (by_col ? kUnitCol : kUnitOne), E5>(t, su, ru, packed);

  if (!TRANS)
    store_patch(packed, a.codes, a.ldc, a.rows, a.cols, row0, c);
  else
    store_patch_transposed(packed, lds_t, a.codes, a.ldc, a.rows, a.cols, r0, c0);

  // scales of the block granularities (TENSOR / ROW / COL are finalized later)
  if (K == kBlock1x128) {
    // output index (c / 128) * rows + r, the same for the transposed layout;
    // lane cc < 8 of a row group holds the scale of the thread's row cc
    const int64_t r = row0 + cc;
    if (cc < 8 && r < a.rows && c < a.cols) a.scales[(c >> 7) * a.rows + r] = mine.s;
  } else if (K == kBlock128x1) {
    // output index (r0 / 128) * cols + c, the same for the transposed layout;
    // thread (rg < 8, cc) holds column 8 cc + rg's scale
    const int64_t cj = c0 + cc * 8 + rg;
    if (rg < 8 && cj < a.cols) a.scales[tr * a.cols + cj] = mine.s;
  } else if (K == kBlock128x128) {
    if (threadIdx.x == 0) {
      const int64_t idx = TRANS ? tc * tiles_r + tr : tr * tiles_c + tc;
      a.scales[idx] = mine.s;
    }
  }
}

// Both operand layouts of the backward pass from one read.  A 128 x 128
// tile is quantized twice: per 1x128 unit (its rows), with codes stored as
// read and scales at (c / 128) * rows + r, and per 128x1 unit (its
// columns), with codes stored transposed, codes_t[c][r], and scales at
// (r / 128) * cols + c.  Each half is the single-layout kernel's work, so
// each result is byte-identical to it.
template <bool E5>
__global__ __launch_bounds__(kThreads) void quant_dual_kernel(DualArgs d) {
  __shared__ float lds_red[4 * kTile];
  __shared__ uint64_t lds_t[kTile * kTile / 8];
  const QuantArgs& a = d.a;
  const int cc = threadIdx.x & 15, rg = threadIdx.x >> 4;
  const int64_t tr = blockIdx.y;
  const int64_t r0 = tr * kTile, c0 = (int64_t)blockIdx.x * kTile;
  const int64_t row0 = r0 + rg * 8, c = c0 + cc * 8;

  Tile t;
  load_patch(a, row0, c, t);
  uint32_t packed[8][2];
  UnitScale mine;
  float su[8], ru[8];

  share_row_units<E5>(block_row_amax(t), a.pow2 != 0, mine, su, ru);
  encode_patch<kUnitRow, E5>(t, su, ru, packed);
  store_patch(packed, a.codes, a.ldc, a.rows, a.cols, row0, c);
  {
    const int64_t r = row0 + cc;
    if (cc < 8 && r < a.rows && c < a.cols) a.scales[(c >> 7) * a.rows + r] = mine.s;
  }

  float m[8];
  tile_col_max(t, lds_red, m);
  float amax = m[0];
#pragma unroll
  for (int j = 1; j < 8; ++j) amax = (rg & 7) == j ? m[j] : amax;
  share_col_units<E5>(amax, a.pow2 != 0, lds_red, mine, su, ru);
  encode_patch<kUnitCol, E5>(t, su, ru, packed);
  store_patch_transposed(packed, lds_t, d.codes_t, d.ldc_t, a.rows, a.cols, r0, c0);
  const int64_t cj = c0 + cc * 8 + rg;
  if (rg < 8 && cj < a.cols) d.scales_t[tr * a.cols + cj] = mine.s;
}

// Partial maxima of the multi-tile granularities: float i sits at float
// i % per of line i / per, lines being `ld` bytes apart.  In the code array
// a line is one of its rows (columns when transposed) and holds per = its
// length / 4 floats, so nothing outside the codes themselves is written; in
// `scales` (one partial per unit) it is one line.
struct Partials {
  uint8_t* base;
  int64_t per, ld;
  __device__ __forceinline__ float* at(int64_t i) const {
    return reinterpret_cast<float*>(base + (i / per) * ld) + (i % per);
  }
};

// Amax pass of COL and of ROW with transposed output, per 128 x 128 tile:
// the partial of row r in tile column tc at tc * rows + r, of column c in
// tile row tr at tr * cols + c.
template <int K>
__global__ __launch_bounds__(kThreads) void amax_tile_kernel(QuantArgs a, Partials part) {
  __shared__ float lds_red[4 * kTile];
  const int cc = threadIdx.x & 15, rg = threadIdx.x >> 4;
  const int64_t r0 = (int64_t)blockIdx.y * kTile;
  const int64_t c0 = (int64_t)blockIdx.x * kTile;
  Tile t;
  load_patch(a, r0 + rg * 8, c0 + cc * 8, t);
  if (K == kPreRow) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float m = row16_max(row_partial_max(t, i));
      const int64_t r = r0 + rg * 8 + i;
      if (cc == 0 && r < a.rows) *part.at((int64_t)blockIdx.x * a.rows + r) = m;
    }
  } else {
    float m[8];
    tile_col_max(t, lds_red, m);
    const int64_t c = c0 + cc * 8;  // cols % 16 == 0: all eight columns or none
    if (rg == 0 && c < a.cols) {
#pragma unroll
      for (int j = 0; j < 8; ++j) *part.at((int64_t)blockIdx.y * a.cols + c + j) = m[j];
    }
  }
}

// S of each unit from its partials (those of unit u at u, u + units, ...):
// a workgroup takes 64 units and its sixteen waves split the partials,
// eight loads in flight per lane at a time (a column's 128 partials of a
// 16384-row input are then one round of loads, not a chain of 32), and LDS
// joins the waves.  A max is exact in any order.
constexpr int kReduceWaves = 16, kReduceDepth = 8;

template <bool E5>
__global__ __launch_bounds__(kReduceWaves * 64) void reduce_units_kernel(Partials part, int64_t units,
                                                                        int64_t nparts, float* scales, int pow2) {
  __shared__ float lds[kReduceWaves][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t u = (int64_t)blockIdx.x * 64 + lane;
  float m = 0.0f;
  if (u < units) {
    for (int64_t p0 = wave; p0 < nparts; p0 += kReduceWaves * kReduceDepth) {
      float v[kReduceDepth];
#pragma unroll
      for (int j = 0; j < kReduceDepth; ++j) {
        const int64_t pj = p0 + (int64_t)kReduceWaves * j;
        v[j] = pj < nparts ? *part.at(pj * units + u) : 0.0f;
      }
#pragma unroll
      for (int j = 0; j < kReduceDepth; ++j) m = fmaxf(m, v[j]);
    }
  }
  lds[wave][lane] = m;
  __syncthreads();
  if (wave == 0 && u < units) {
#pragma unroll
    for (int w = 1; w < kReduceWaves; ++w) m = fmaxf(m, lds[w][lane]);
    scales[u] = unit_scale_fmt<E5>(m, pow2 != 0).s;
  }
}

// S of TENSOR from the nparts partials of its amax pass (one workgroup).
template <bool E5>
__global__ __launch_bounds__(256) void reduce_tensor_kernel(Partials part, int64_t nparts, float* scales, int pow2) {
  __shared__ float lds4[4];
  float m = 0.0f;
  for (int64_t p = threadIdx.x; p < nparts; p += 256) m = fmaxf(m, *part.at(p));
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) lds4[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0)
    scales[0] = unit_scale_fmt<E5>(fmaxf(fmaxf(lds4[0], lds4[1]), fmaxf(lds4[2], lds4[3])), pow2 != 0).s;
}

// ROW units without transposition, in one pass over memory: a wave takes
// one row at a time.  Lane l holds the 16-byte pieces l, l + 64, ... of a
// 4096-element chunk of the row, so each load instruction reads 1 KB of it,
// and the row's amax is a wave reduction.  A row of more than 4096 elements
// is walked twice, the second time out of L2: for its amax, then for its
// codes.
constexpr int kRowChunk = 4096;
constexpr int kRowWaves = 4;

__device__ __forceinline__ void load_row_chunk(const QuantArgs& a, const uint16_t* xr, int64_t c0, Tile& t) {
  const int lane = threadIdx.x & 63;
  uint4 w[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int64_t c = c0 + q * 512 + lane * 8;
    w[q] = make_uint4(0u, 0u, 0u, 0u);
    if (c < a.cols) w[q] = *reinterpret_cast<const uint4*>(xr + c);
  }
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    t.v[q][0] = bf16_lo(w[q].x);
    t.v[q][1] = bf16_hi(w[q].x);
    t.v[q][2] = bf16_lo(w[q].y);
    t.v[q][3] = bf16_hi(w[q].y);
    t.v[q][4] = bf16_lo(w[q].z);
    t.v[q][5] = bf16_hi(w[q].z);
    t.v[q][6] = bf16_lo(w[q].w);
    t.v[q][7] = bf16_hi(w[q].w);
  }
}

template <bool E5>
__global__ __launch_bounds__(kRowWaves * 64) void quant_row_kernel(QuantArgs a) {
  const int lane = threadIdx.x & 63;
  const bool one_chunk = a.cols <= kRowChunk;
  const int64_t stride = (int64_t)gridDim.x * kRowWaves;
  for (int64_t r = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6); r < a.rows; r += stride) {
    const uint16_t* xr = a.x + r * a.ldx;
    Tile t;
    float m = 0.0f;
    for (int64_t c0 = 0; c0 < a.cols; c0 += kRowChunk) {
      load_row_chunk(a, xr, c0, t);
#pragma unroll
      for (int q = 0; q < 8; ++q) m = fmaxf(m, row_partial_max(t, q));
    }
    const UnitScale u = unit_scale_fmt<E5>(wave_max(m), a.pow2 != 0);
    float su[8], ru[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      su[i] = u.s;
      ru[i] = u.r;
    }
    for (int64_t c0 = 0; c0 < a.cols; c0 += kRowChunk) {
      if (!one_chunk) load_row_chunk(a, xr, c0, t);
      uint32_t packed[8][2];
      encode_patch<kUnitOne, E5>(t, su, ru, packed);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int64_t c = c0 + q * 512 + lane * 8;
        if (c < a.cols) *reinterpret_cast<uint2*>(a.codes + r * a.ldc + c) = make_uint2(packed[q][0], packed[q][1]);
      }
    }
    if (lane == 0) a.scales[r] = u.s;
  }
}

// Amax pass of TENSOR: a grid-stride walk over 32 x 512 tiles (1 KB row
// pieces per load instruction) keeping a running max per thread; workgroup
// b writes its maximum as partial b.
__global__ __launch_bounds__(kThreads) void amax_tensor_kernel(QuantArgs a, Partials part) {
  __shared__ float lds4[4];
  const int64_t tiles_c = (a.cols + kWideCols - 1) / kWideCols;
  const int64_t tiles = tiles_c * ((a.rows + kWideRows - 1) / kWideRows);
  float m = 0.0f;
  for (int64_t t = blockIdx.x; t < tiles; t += gridDim.x) {
    const int64_t r0 = (t / tiles_c) * kWideRows, c0 = (t % tiles_c) * kWideCols;
    Tile p;
    load_patch(a, r0 + (threadIdx.x >> 6) * 8, c0 + ((threadIdx.x >> 4) & 3) * 128 + (threadIdx.x & 15) * 8, p);
#pragma unroll
    for (int i = 0; i < 8; ++i) m = fmaxf(m, row_partial_max(p, i));
  }
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) lds4[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) *part.at(blockIdx.x) = fmaxf(fmaxf(lds4[0], lds4[1]), fmaxf(lds4[2], lds4[3]));
}

template <bool E5>
__global__ void cast_f32_kernel(const float* x, int64_t n, float scale, uint8_t* codes) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const float q = x[i] / scale;  // IEEE division: any fp32 x and scale
    codes[i] = (uint8_t)(fp8_pack2<E5, false>(q, q, 0u) & 0xffu);
  }
}

template <int K, bool TRANS, bool E5>
hipError_t launch_tile(const QuantArgs& a, hipStream_t s) {
  constexpr bool kWide = !TRANS && (K == kBlock1x128 || K == kPreRow || K == kPreTensor);
  constexpr int64_t tr = kWide ? kWideRows : kTile, tc = kWide ? kWideCols : kTile;
  const dim3 grid((unsigned)((a.cols + tc - 1) / tc), (unsigned)((a.rows + tr - 1) / tr));
  quant_tile_kernel<K, TRANS, E5><<<grid, kThreads, 0, s>>>(a);
  return hipGetLastError();
}

// Workgroups of the TENSOR amax pass (each writes one partial).
constexpr int64_t kTensorParts = 1024;

// TENSOR, COL and ROW with transposed output: partial amaxes, their
// reduction to S, then the cast.
template <int K, bool E5>
hipError_t launch_two_pass(const QuantArgs& a, bool trans, hipStream_t s) {
  // the code array as lines of floats (rows % 16 == 0 when transposed,
  // cols % 16 == 0 always)
  Partials in_codes{a.codes, (trans ? a.rows : a.cols) / 4, a.ldc};
  Partials in_scales{reinterpret_cast<uint8_t*>(a.scales), INT64_MAX, 0};
  hipError_t e;
  if (K == kPreTensor) {
    const int64_t tiles = ((a.cols + kWideCols - 1) / kWideCols) * ((a.rows + kWideRows - 1) / kWideRows);
    const int64_t parts = tiles < kTensorParts ? tiles : kTensorParts;  // <= rows * cols / 4: they fit
    amax_tensor_kernel<<<(unsigned)parts, kThreads, 0, s>>>(a, in_codes);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    reduce_tensor_kernel<E5><<<1, 256, 0, s>>>(in_codes, parts, a.scales, a.pow2);
  } else {
    const int64_t tiles_r = (a.rows + kTile - 1) / kTile, tiles_c = (a.cols + kTile - 1) / kTile;
    const int64_t units = K == kPreRow ? a.rows : a.cols, nparts = K == kPreRow ? tiles_c : tiles_r;
    // one partial per unit: in place in `scales`; else nparts <= (its
    // dimension) / 4 (it exceeds 128 and so 4 nparts), and the codes hold
    // rows * cols / 4 floats
    const Partials part = nparts == 1 ? in_scales : in_codes;
    const dim3 grid((unsigned)tiles_c, (unsigned)tiles_r);
    amax_tile_kernel<K><<<grid, kThreads, 0, s>>>(a, part);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    reduce_units_kernel<E5><<<(unsigned)((units + 63) / 64), kReduceWaves * 64, 0, s>>>(part, units, nparts, a.scales,
                                                                                       a.pow2);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return trans ? launch_tile<K, true, E5>(a, s) : launch_tile<K, false, E5>(a, s);
}

template <bool E5>
hipError_t launch_quantize_fmt(const QuantArgs& a, int granularity, bool trans, int64_t nscales, hipStream_t s) {
  (void)nscales;
  switch (granularity) {
    case 3: return trans ? launch_tile<kBlock1x128, true, E5>(a, s) : launch_tile<kBlock1x128, false, E5>(a, s);
    case 4: return trans ? launch_tile<kBlock128x1, true, E5>(a, s) : launch_tile<kBlock128x1, false, E5>(a, s);
    case 5:
      return trans ? launch_tile<kBlock128x128, true, E5>(a, s) : launch_tile<kBlock128x128, false, E5>(a, s);
    case 0: return launch_two_pass<kPreTensor, E5>(a, trans, s);
    case 1: {
      if (trans) return launch_two_pass<kPreRow, E5>(a, trans, s);
      const int64_t blocks = (a.rows + kRowWaves - 1) / kRowWaves;
      quant_row_kernel<E5><<<(unsigned)(blocks < 16384 ? blocks : 16384), kRowWaves * 64, 0, s>>>(a);
      return hipGetLastError();
    }
    case 2: return launch_two_pass<kPreCol, E5>(a, trans, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace quant_detail

using namespace quant_detail;

hipError_t launch_quantize(const QuantArgs& a, int granularity, bool trans, int64_t nscales, hipStream_t s) {
  return a.e5m2 ? launch_quantize_fmt<true>(a, granularity, trans, nscales, s)
                : launch_quantize_fmt<false>(a, granularity, trans, nscales, s);
}

hipError_t launch_quantize_dual(const DualArgs& d, hipStream_t s) {
  const dim3 grid((unsigned)((d.a.cols + kTile - 1) / kTile), (unsigned)((d.a.rows + kTile - 1) / kTile));
  if (d.a.e5m2)
    quant_dual_kernel<true><<<grid, kThreads, 0, s>>>(d);
  else
    quant_dual_kernel<false><<<grid, kThreads, 0, s>>>(d);
  return hipGetLastError();
}

hipError_t launch_cast_f32(const float* x, int64_t n, float scale, bool e5m2, uint8_t* codes, hipStream_t s) {
  const int64_t blocks = (n + 255) / 256;
  const unsigned grid = (unsigned)(blocks < 8192 ? blocks : 8192);
  if (e5m2)
    cast_f32_kernel<true><<<grid, 256, 0, s>>>(x, n, scale, codes);
  else
    cast_f32_kernel<false><<<grid, 256, 0, s>>>(x, n, scale, codes);
  return hipGetLastError();
}

}  // namespace fp8q
