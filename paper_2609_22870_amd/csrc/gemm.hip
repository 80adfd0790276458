// Scaled FP8 GEMM of the FP8 linear layer on gfx950:
//   C[m][n] = sum_k (S_A(m,k) A[m][k]) (S_B(n,k) B[n][k]),  A, B OCP E4M3,
// fp32 accumulation on the matrix cores, bf16 output.
//
// Tiling: a workgroup owns a BM x BN tile of C and steps K by 128, which is
// both the depth of one v_mfma_f32_16x16x128_f8f6f4 and the length of one
// scale block, so a blockwise step is one MFMA per 16 x 16 tile into a
// zeroed partial, then one FMA per accumulator that adds S_A * S_B * P.
// Four shapes are built: 256 x 256 tiles with eight waves of 128 x 64 (the
// large-problem kernel: 64 FP8 bytes of LDS traffic per MFMA instead of
// 128), 128 x 128 tiles with four waves of 64 x 64 (small grids, and the
// (1x128, 1x128) pair whose per-column B scales need more registers), and
// for skinny problems such as a decode step, 128 x 128 tiles with eight
// waves of 32 x 64 and 64 x 64 tiles with four waves of 32 x 32, where a
// few tiles split their K blocks over two groups of waves.
//
// Operand tiles (rows x 128 bytes of K) go global -> LDS with the
// direct-to-LDS 16-byte buffer loads of gfx950 (no VGPR staging), in a ring
// of stages, XOR-swizzled against LDS bank conflicts; the scale vectors of a
// step travel the same way.  Workgroups are rastered so that the tiles
// running together on one XCD (which has its own L2) share operand rows.
// The MFMA "A" operand is the B tile (rows n) and the MFMA "B" operand the A
// tile (rows m): each lane then ends with four consecutive n of one m.  The
// epilogue rounds to bf16 and stages the C tile through LDS so that it
// leaves in 16-byte row segments.
#include <type_traits>

#include "device_common.h"
#include "internal.h"

namespace fp8q {

namespace gemm_detail {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef unsigned int v2u __attribute__((ext_vector_type(2)));

constexpr int kBK = 128;
constexpr int kGroupM = 8;  // tile rows per group of the raster

typedef __attribute__((address_space(3))) void lds_void;

// Operand formats of a GEMM: bit 0 set when A's codes are E5M2, bit 1 when
// B's are (else E4M3).  B's tile is the instruction's first operand and A's
// its second, so B's format goes to the first format field (cbsz) and A's to
// the second (blgp); 0 selects E4M3 (fp8), 1 E5M2 (bf8).
template <int FMT>
__device__ __forceinline__ v4f mfma_16x16x128(const v8i& a, const v8i& b, const v4f& c) {
  // Scale operands 0 select the unscaled instruction.
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, (FMT >> 1) & 1, FMT & 1, 0, 0, 0, 0);
}

// The same with power-of-two block scales applied inside the instruction:
// scale_a (of this lane) multiplies row l % 16 of `a` over its 32-deep K
// piece l / 16, scale_b the same of `b`; each is an E8M0 byte (2^(e - 127),
// e = 127 for 1.0; measured on gfx950 with runtime operands).
__device__ __forceinline__ v4f mfma_16x16x128_e8(const v8i& a, const v8i& b, const v4f& c, int scale_a,
                                                 int scale_b) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, scale_a, 0, scale_b);
}

// E8M0 byte of a power-of-two fp32 scale in [2^-127, 2^127]: its exponent
// field (2^-127, an fp32 subnormal, has field 0, which E8M0 reads as 2^-127).
__device__ __forceinline__ int e8m0_of(float pow2) { return (int)((__float_as_uint(pow2) >> 23) & 0xffu); }

typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

// Two floats to two bf16 (round to nearest even), packed low then high: one
// v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((v2f{lo, hi}), v2bf));
}

// Buffer resource over `bytes` bytes at `base` (gfx9 raw buffer: stride 0,
// loads past `bytes` return zero, stores past it are dropped).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ float load_f32(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

// LDS placement of the operand tiles.  Tile row r (128 bytes of K) sits at
// byte 128 r; its logical 16-byte chunk c sits at physical chunk
// c ^ chunk_swizzle(r).  The MFMA fragment reads (ds_read_b128) have lane l
// read row l % 16 of a strip at logical chunk 2 (l / 16) + h.  Measured on
// gfx950 (64 banks of 4 bytes): a ds_read_b128 goes out in four passes of
// 16 lanes, a pass being the lanes that agree in lane bit 5 and in the
// parity of lane bits 2..4, and a pass takes one cycle when its 16 lanes hit
// 16 different 16-byte bank groups (address bits 4..7), two when two lanes
// share one, and so on.  The bank group of a fragment read is
// (row bit 0, c ^ chunk_swizzle(row)); with chunk_swizzle(r) = r1 + 6 r2
// (bits 1 and 2 of r) the 16 lanes of every pass land on 16 different
// groups, for both halves h.  (c ^ ((r >> 1) & 7), the swizzle that suits
// sixteen consecutive lanes, measured two-way conflicted.)
// Calls f(integral_constant<int, I>) for I = 0 .. N-1, unrolled.
template <int N, typename F, int I = 0>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, F, I + 1>(static_cast<F&&>(f));
  }
}

__device__ __forceinline__ int chunk_swizzle(int r) { return ((r >> 1) & 1) | (((r >> 2) & 1) * 6); }

// Copies of ROWS x 128-byte operand tiles (K bytes k0 .. k0+127) into LDS
// with direct buffer-to-LDS loads, in the placement above.  A wave
// instruction moves a group of eight rows: lane l lands at byte 16 l of the
// group's 1 KB, i.e. row l / 8, physical chunk l % 8, so it fetches the
// logical chunk that maps there.  Each
// lane keeps one 32-bit row offset per group; rows past the operand read as
// zero through the buffer bounds (their results are never stored).
template <int ROWS, int NWAVES>
struct TileLoader {
  static constexpr int kGroups = ROWS / 8;
  static constexpr int kPerWave = kGroups / NWAVES;
  static_assert(kGroups % NWAVES == 0, "row groups must split evenly over the waves");
  static_assert(kPerWave % 2 == 0, "groups come in pairs (the swizzle repeats every 16 rows)");
  __amdgpu_buffer_rsrc_t rsrc;
  int off_even, off_odd;  // this lane's offset for the wave's first group, and the second
  int step;               // byte distance between groups g and g+2 (16 rows)

  __device__ __forceinline__ TileLoader(const uint8_t* base, int64_t ld, int64_t row0, int64_t rows, int wave) {
    rsrc = make_rsrc(base, (uint32_t)(rows * ld));
    const int lane = threadIdx.x & 63;
    const int trow = wave * kPerWave * 8 + (lane >> 3);  // tile row of group 0 (kPerWave even)
    // the chunk swizzle repeats every 16 rows: even groups share one value,
    // odd groups another
    const int chunk_even = (lane & 7) ^ chunk_swizzle(trow);
    const int chunk_odd = (lane & 7) ^ chunk_swizzle(trow + 8);
    const int64_t r = row0 + trow;
    // rows past the operand give offsets past the buffer: they read zero
    off_even = (int)(r * ld) + chunk_even * 16;
    off_odd = (int)((r + 8) * ld) + chunk_odd * 16;
    step = (int)(16 * ld);
  }

  // the wave's row group G (of kPerWave)
  template <int G>
  __device__ __forceinline__ void load_group(int k0, uint8_t* lds_tile, int wave) const {
    const int off = (G & 1 ? off_odd : off_even) + (G >> 1) * step;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)(lds_tile + (wave * kPerWave + G) * 1024), 16, off,
                                             k0, 0, 0);
  }
  __device__ __forceinline__ void load(int k0, uint8_t* lds_tile, int wave) const {
    static_for<kPerWave>([&](auto g) { load_group<decltype(g)::value>(k0, lds_tile, wave); });
  }
};

typedef __attribute__((address_space(3))) uint8_t lds_u8;

__device__ __forceinline__ uint32_t lds_addr(const uint8_t* p) {
  return (uint32_t)(uintptr_t)(const lds_u8*)p;
}

// Issue the reads of 32 K-bytes of one operand row for the MFMA: logical
// chunks 2g and 2g+1 of tile row `row` (g = lane / 16), un-swizzled.  The
// reads are inline asm: the compiler then sees no LDS load it would have to
// order after the direct-to-LDS loads still in flight for the next stage (it
// would otherwise wait for all of them before every step).  The data is
// ready only after a later lds_wait naming the fragment.
//
// Because the compiler does not see these as register writes, two rules
// keep them clear of matrix instructions that may still be reading their
// sources: the destination is early-clobber against `busy` and `busy2`,
// fragments of MFMAs possibly in flight or still to be issued (so it never
// takes those registers), and the
// reads take `after` as an input, a VALU result computed from the output of
// the last MFMA whose source registers may be reused (so that MFMA is done
// before they issue).  (Making the addresses themselves depend on it, by an
// empty asm that rewrites them, cost two register copies per read.)
//
// Fragment rows come in strips of 16 (row = strip base + lane % 16), so the
// swizzle term chunk_swizzle(row) depends on the lane only: the two chunk
// addresses are a per-lane constant `lane_off` (low, high) plus the strip's
// byte offset `imm` (a multiple of 2 KB), which goes into the instruction.
struct FragAddr {
  uint32_t lo, hi;  // LDS byte addresses of this lane's two chunks in strip 0
};

__device__ __forceinline__ FragAddr frag_addr(const uint8_t* lds_tile_strip0) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15, sw = chunk_swizzle(r);
  const uint32_t base = lds_addr(lds_tile_strip0) + r * 128;
  return FragAddr{base + (((2 * g) ^ sw) << 4), base + (((2 * g + 1) ^ sw) << 4)};
}

template <int IMM>
__device__ __forceinline__ v8i read_frag(FragAddr a, const v8i& busy, const v8i& busy2, float after) {
  uint4 lo, hi;
  asm volatile("ds_read_b128 %0, %2 offset:%4\n\tds_read_b128 %1, %3 offset:%4"
               : "=&v"(lo), "=&v"(hi)
               : "v"(a.lo), "v"(a.hi), "i"(IMM), "v"(busy), "v"(busy2), "v"(after));
  v8i f;
  f[0] = (int)lo.x; f[1] = (int)lo.y; f[2] = (int)lo.z; f[3] = (int)lo.w;
  f[4] = (int)hi.x; f[5] = (int)hi.y; f[6] = (int)hi.z; f[7] = (int)hi.w;
  return f;
}

// Scalar and 4-wide fp32 reads from LDS, completed by the next lds_wait
// (the values may only be used after it).
__device__ __forceinline__ float lds_read_f32(uint32_t addr, int imm) {
  float v;
  asm volatile("ds_read_b32 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(imm));
  return v;
}
__device__ __forceinline__ void lds_read_f32x4(uint32_t addr, float (&v)[4]) {
  float4 t;
  asm volatile("ds_read_b128 %0, %1" : "=v"(t) : "v"(addr));
  v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
}

// Wait until at most N LDS reads of this wave are outstanding, and make
// `f` (whose reads were issued before the last N) count as written here.
// The loop issues no scalar memory loads, so LDS reads retire in order.
template <int N>
__device__ __forceinline__ void lds_wait(v8i& f) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(f) : "n"(N));
}

// No instruction may be scheduled across this point: it pins the matrix
// instructions next to the (inline asm) LDS waits they depend on.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

template <int N>
__device__ __forceinline__ void lds_wait2(v8i& f, v8i& h) {
  asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(f), "+v"(h) : "n"(N));
}

__device__ __forceinline__ void wait_vmem_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// at most N vector-memory instructions of this wave still in flight
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }


// Empty asm that claims to read `done` and rewrite `next`: whatever consumes
// `next` afterwards is ordered after everything that produced `done`.
template <int TJ>
__device__ __forceinline__ void order_after(v8i& next, v4f (&done)[TJ]) {
  asm volatile("" : "+v"(next) : "v"(done[0]), "v"(done[TJ - 1]));
  if (TJ > 2) asm volatile("" : "+v"(next) : "v"(done[1]), "v"(done[TJ > 2 ? 2 : 0]));
}

// Tile coordinates of this workgroup.  Workgroup b runs on XCD b % 8, so
// each XCD is given a contiguous range of the raster (sharing its L2), and
// the raster walks kGroupM tile rows at a time so that consecutive tiles
// reuse A rows and B rows.
__device__ __forceinline__ int xcd_order(int total, int b) {
  const int xcd = b & 7, per = total >> 3, extra = total & 7;
  return xcd * per + (xcd < extra ? xcd : extra) + (b >> 3);
}

// Tile (tm, tn) at position id of a problem's raster.  A group of kGroupM
// tile rows streams the whole B operand past the L2s once per group, and A
// only once in all; when the two operands together overflow the 256 MB
// last-level cache, those repeated passes over B come from HBM, so if B is
// the larger operand the raster walks groups of kGroupM tile columns
// instead (the 32B up-projection's wgrad: A 84 MB, B 419 MB).  The mapping
// decides only which workgroup computes which tile: each output element's
// K order is fixed by its column.
constexpr int64_t kLastLevelCache = 256ll << 20;
template <int BM, int BN>
__device__ __forceinline__ void raster(int64_t M, int64_t N, int64_t K, int id, int& tm, int& tn) {
  const int tiles_m = (int)((M + BM - 1) / BM), tiles_n = (int)((N + BN - 1) / BN);
  const bool col_groups = N > M && tiles_m > kGroupM && (M + N) * K > kLastLevelCache;
  const int grouped = col_groups ? tiles_n : tiles_m;  // tiles across the groups
  const int walked = col_groups ? tiles_m : tiles_n;   // tiles along one group
  const int per_group = kGroupM * walked;
  const int group = id / per_group;
  const int first = group * kGroupM;
  const int gsize = (grouped - first) < kGroupM ? (grouped - first) : kGroupM;
  const int in_group = id - group * per_group;
  const int across = first + in_group % gsize, along = in_group / gsize;
  tm = col_groups ? along : across;
  tn = col_groups ? across : along;
}

template <int BM, int BN>
__device__ __forceinline__ void tile_coords(int64_t M, int64_t N, int64_t K, int b, int& tm, int& tn) {
  const int total = (int)((M + BM - 1) / BM) * (int)((N + BN - 1) / BN);
  raster<BM, BN>(M, N, K, xcd_order(total, b), tm, tn);
}

// Quantized output: the tile's bf16 C, staged in LDS (row m at byte m *
// ROW_BYTES, 16-byte chunk c at chunk c ^ (m & CHUNK_MASK)), quantized per
// 1x128 unit along N by Eq. 3, exactly as the quantizer would quantize the
// bf16 output: codes [M][ldq], scales [N/128][cs_ld] (the quantizer's 1x128
// layout).  A thread takes chunk c (eight columns) of rows mt0 + p * RPP for
// the PASSES passes p; the 16 chunks of one row's 128-column unit sit in the
// 16 lanes of a DPP row, so a unit's amax is a DPP row max.  Lane j of the
// DPP row then computes the S and 1/S of pass j's unit (two IEEE divisions
// per lane, not per pass) and the lanes exchange them by shuffles.
template <int PASSES, int ROW_BYTES, int CHUNK_MASK, int RPP>
__device__ __forceinline__ void store_quantized(const GemmArgs& g, const uint8_t* lds, int64_t m0, int64_t n0,
                                                int chunks_per_row) {
  static_assert(PASSES <= 16, "one pass per lane of a DPP row");
  const int lane = threadIdx.x & 63, j = lane & 15;
  const int c = threadIdx.x % chunks_per_row, mt0 = threadIdx.x / chunks_per_row;
  const int64_t n = n0 + c * 8;
  uint4 v[PASSES];
  float am[PASSES];
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int mt = mt0 + p * RPP;
    v[p] = *reinterpret_cast<const uint4*>(lds + mt * ROW_BYTES + ((c ^ (mt & CHUNK_MASK)) << 4));
    const uint32_t w[4] = {v[p].x, v[p].y, v[p].z, v[p].w};
    float m = 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) m = fmaxf(m, fmaxf(fabsf(bf16_lo(w[e])), fabsf(bf16_hi(w[e]))));
    am[p] = row16_max(m);
  }
  float amax = am[0];
#pragma unroll
  for (int p = 1; p < PASSES; ++p) amax = j == p ? am[p] : amax;
  const UnitScale mine = unit_scale(amax);
  const bool fast = __all(j >= PASSES || mine.fast);
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const float s = __shfl(mine.s, (lane & 48) | p, 64), r = __shfl(mine.r, (lane & 48) | p, 64);
    const UnitScale u{s, r, s >= 0x1p-90f};
    const uint32_t w[4] = {v[p].x, v[p].y, v[p].z, v[p].w};
    float q[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = bf16_lo(w[e]), hi = bf16_hi(w[e]);
      q[2 * e] = fast ? fast_quotient(lo, s, r) : quotient(lo, u);
      q[2 * e + 1] = fast ? fast_quotient(hi, s, r) : quotient(hi, u);
    }
    const uint32_t c0 = e4m3_pack2<true>(q[2], q[3], e4m3_pack2<false>(q[0], q[1], 0u));
    const uint32_t c1 = e4m3_pack2<true>(q[6], q[7], e4m3_pack2<false>(q[4], q[5], 0u));
    const int64_t m = m0 + mt0 + p * RPP;
    if (m < g.M && n < g.N) *reinterpret_cast<uint2*>(g.Cq + m * g.ldq + n) = make_uint2(c0, c1);
  }
  const int64_t m = m0 + mt0 + j * RPP;
  if (j < PASSES && m < g.M && n < g.N) g.Cs[(n >> 7) * g.cs_ld + m] = mine.s;
}

// Split-K reduction.  The g.splits workgroups of one tile each hold the
// fp32 partial tile of their K range.  Each writes it to its slot of the
// workspace (slot s of tile t at part + (t * splits + s) * BM * BN floats,
// every wave's accumulators in register order, lane-interleaved in pairs),
// then counts itself in cnt[t].  The workgroup that counts last reads all
// the slots back and adds the partials in split order, ((p0 + p1) + p2) +
// ..., so the sum does not depend on the order of arrival; it resets
// cnt[t] to zero for the next call and goes on to the
// epilogue, the others end.  Visibility across XCDs (each with its own L2)
// without writing back or invalidating the L2s: the partials are stored
// and loaded with agent-scope accesses (coherent at the device level), the
// stores are complete before the count (s_waitcnt), and the loads go out
// only after the count that found them all.  Returns true in the last
// workgroup (then `acc` holds the sum).
template <int TI, int TJ, int TILE_FLOATS>
__device__ __forceinline__ bool splitk_reduce(const GemmArgs& g, v4f (&acc)[TI][TJ], int split, int tile, int wave,
                                              int lane, uint8_t* flag_lds) {
  constexpr int kPairs = TI * TJ * 2;  // 64-bit pairs of accumulators per lane
  const int S = g.splits;
  uint64_t* const slab = reinterpret_cast<uint64_t*>(g.part + (int64_t)tile * S * TILE_FLOATS);
  constexpr int64_t slot_pairs = TILE_FLOATS / 2;
  auto at = [&](int s, int q) { return slab + s * slot_pairs + ((int64_t)wave * kPairs + q) * 64 + lane; };
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint64_t v = (uint64_t)__float_as_uint(acc[i][j][2 * h]) |
                           ((uint64_t)__float_as_uint(acc[i][j][2 * h + 1]) << 32);
        __hip_atomic_store(at(split, (i * TJ + j) * 2 + h), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's partial is stored
  __syncthreads();                                   // and every wave's
  __attribute__((address_space(3))) uint32_t* const flag = (__attribute__((address_space(3))) uint32_t*)flag_lds;
  if (threadIdx.x == 0) {
    const uint32_t before = __hip_atomic_fetch_add(g.cnt + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const bool last = before == (uint32_t)(S - 1);
    if (last) __hip_atomic_store(g.cnt + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *flag = last ? 1u : 0u;
  }
  __syncthreads();
  if (*flag == 0u) return false;
  // every slot is read back (this workgroup's own too: the same bits it
  // holds), four at a time with all their loads in flight, and added in
  // split order; slots past S repeat the last one and are not added
  v4f sum[TI][TJ];
  for (int s0 = 0; s0 < S; s0 += 4) {
    v4f p[4][TI][TJ];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int s = s0 + u < S ? s0 + u : S - 1;
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint64_t v = __hip_atomic_load(at(s, (i * TJ + j) * 2 + h), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            p[u][i][j][2 * h] = __uint_as_float((uint32_t)v);
            p[u][i][j][2 * h + 1] = __uint_as_float((uint32_t)(v >> 32));
          }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (s0 + u < S) {
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int j = 0; j < TJ; ++j) sum[i][j] = s0 + u == 0 ? p[u][i][j] : sum[i][j] + p[u][i][j];
      }
    }
  }
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = sum[i][j];
  return true;
}

// One workgroup computes a BM x BN tile of C with (BM/WM) x (BN/WN) waves,
// each owning WM x WN as (WM/16) x (WN/16) MFMA tiles of 16 x 16.  QOUT: the
// tile leaves as E4M3 codes and 1x128 scales of its bf16 values (see
// store_quantized) instead of bf16.
// KS > 1 (skinny problems, 64 x 64 tiles): KS groups of waves share the
// tile, group k taking the K blocks k, k + KS, ... with its own LDS ring;
// their partial tiles are summed in LDS at the end, group 1 into group 0,
// then group 2, ... (a fixed order).  Each group's step chain (barrier,
// fragment reads, MFMAs, FMAs) then overlaps the others' on the same SIMDs.
// SPLITK: the workgroup is split `split` of the g.splits that share tile
// number `tile`, and sums the K blocks split * KT .. split * KT + KT - 1
// (KT = K / 128 / g.splits); see splitk_reduce for how the partial tiles
// meet.
template <int PAIR, int BM, int BN, int WM, int WN, bool QOUT, int FMT, int KS = 1, bool SPLITK = false>
__device__ __forceinline__ void gemm_tile(const GemmArgs& g, int tm, int tn, int split = 0, int tile = 0) {
  constexpr int kWavesN = BN / WN;
  constexpr int kWaves = (BM / WM) * kWavesN;  // waves of one group
  constexpr int TI = WM / 16, TJ = WN / 16;
  constexpr int kTileA = BM * kBK, kTileB = BN * kBK, kStage = kTileA + kTileB;
  // kBlockScaled: per-K-step scale vectors are staged with the tiles;
  // kPromote: they are applied by FMAs on the VALU (fp32 scales), else the
  // accumulation runs in the MFMA accumulator (power-of-two scales enter
  // the instruction itself)
  constexpr bool kBlockScaled = PAIR == kPairBlock || PAIR == kPairBlockK || PAIR == kPairBlockE8;
  constexpr bool kPromote = PAIR == kPairBlock || PAIR == kPairBlockK;
  constexpr bool kWeightBlocks = PAIR == kPairBlock || PAIR == kPairBlockE8;  // B scales per 128 x 128
  // per-step scale vectors of the blockwise pairs, staged like the tiles:
  // A row scales (BM floats) and B scales (the BN/128 weight-block scales,
  // or BN column scales for 1x128 x 1x128)
  constexpr int kScaleA = kBlockScaled ? BM * 4 : 0;
  constexpr int kScaleB = PAIR == kPairBlockK ? BN * 4 : (kWeightBlocks ? 256 : 0);
  constexpr int kScaleStage = kScaleA + kScaleB;
  // LDS ring of kStages operand stages (and their scale vectors): the loads
  // of stage kt + kStages - 1 go out during step kt.  The 256 x 256 tile
  // fits two 64 KB stages; 128 x 128 with four waves of 64 x 64 keeps two
  // (more would cost it its second workgroup per CU); the tiles of skinny
  // problems, whose steps are short next to the load latency, keep four:
  // 64 x 64, and 128 x 128 with eight waves of 32 x 64 (one workgroup per
  // CU).
  constexpr int kStages = (BM >= 128 && WM >= 64) ? 2 : 4;
  static_assert(KS == 1 || (kStages > 2 && !QOUT), "K groups: the 64 x 64 tile");
  constexpr int kGroupBytes = kStages * kStage + kStages * kScaleStage;
  __shared__ __attribute__((aligned(1024))) uint8_t lds_all[KS * kGroupBytes + KS * kWaves * 256];
  const int wave_all = uniform(threadIdx.x >> 6);
  const int kg = KS > 1 ? uniform(wave_all / kWaves) : 0;  // K group
  uint8_t* const lds = lds_all + kg * kGroupBytes;
  uint8_t* const scale_lds = lds + kStages * kStage;
  uint8_t* const dummy_lds = lds_all + KS * kGroupBytes;  // 256 bytes per wave

  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int lane = threadIdx.x & 63;
  const int wave = KS > 1 ? uniform(wave_all % kWaves) : wave_all;  // within the group
  const int wm = (wave / kWavesN) * WM, wn = (wave % kWavesN) * WN;
  // steps of this group (KS divides K / 128) or of this split (g.splits
  // divides it)
  const int KT = (int)(g.K / kBK) / (SPLITK ? g.splits : KS);
  // K block of the group's step st.  Tiles whose first column lies in an
  // odd 1024-column band walk K backwards: the 256 x 256 row-group raster
  // runs 8 tile rows x 4 tile columns (one band) on an XCD at a time and then the next
  // band of the same rows, which so starts on the K blocks of A the last one
  // ended with, still in L2.  Every tile shape takes the same direction for
  // an output element, so a grouped launch sums as a single call would (and
  // so does each sub-problem of a split launch, whose column origins are
  // multiples of 2048 while ldb < 2^20).
  const bool rev = ((n0 >> 10) & 1) != 0;
  auto kb = [&](int st) {
    const int o = rev ? KT - 1 - st : st;
    return SPLITK ? split * KT + o : o * KS + kg;
  };
  const int mw = (int)m0 + wm, nw = (int)n0 + wn;  // wave's first row / column

  v4f acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  // Scales.  This lane accumulates rows m = mw + 16 i + lane % 16 and
  // columns n = nw + 16 j + 4 (lane / 16) + r.  Per K block kt the row
  // scales of A sit at sA[kt * sa_ld + m] (1x128) and the scales of B at
  // sB[(n / 128) * (K / 128) + kt] (128x128) or sB[kt * sb_ld + n] (1x128).
  // The staged scale vectors of a tile cover whole tiles: entries for rows
  // past M (columns past N) repeat the last row's (column's) scale, so that
  // every address stays inside the arrays; they only feed rows or columns
  // that are never stored.
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(g.sA, (uint32_t)(g.sa_count * 4));
  const __amdgpu_buffer_rsrc_t rsB = make_rsrc(g.sB, (uint32_t)(g.sb_count * 4));
  const int kblocks = (int)(g.K / 128);
  // direct-to-LDS loads of the scale vectors of step kt: instruction q moves
  // 64 floats; the A vector takes BM / 64 of them, the B vector the rest.
  // Wave q issues instruction q, without branching: the waves past kQ issue
  // a load whose offset is past the buffer (it reads zeros) into their own
  // 256-byte dummy corner of LDS.
  constexpr int kQA = kScaleA / 256, kQB = kScaleB / 256, kQ = kQA + kQB;
  const bool q_is_a = wave < kQA;
  const __amdgpu_buffer_rsrc_t rs_q = q_is_a ? rsA : rsB;
  int q_dst = 0, q_voff = 0x7fffffff, q_ld = 0, q_base = 0;
  auto scale_offsets = [&]() {  // of the tile at (m0, n0)
    const int last_m = (int)(g.M - 1 - m0), last_n = (int)(g.N - 1 - n0);  // >= 0: the tile is inside C
    if (wave < kQA) {
      q_dst = wave * 256;
      const int r = wave * 64 + lane;
      q_voff = (r < last_m ? r : last_m) * 4;
      q_ld = (int)g.sa_ld * 4;
      q_base = (int)m0 * 4;
    } else if (wave < kQ) {
      q_dst = kScaleA + (wave - kQA) * 256;
      if (kWeightBlocks) {
        // the tile's BN / 128 weight blocks, each with K / 128 scales (the
        // lanes past them read past the array: zeros through the bounds of
        // the vector offset)
        const int nb = (int)(n0 / 128) + (lane < last_n / 128 ? lane : last_n / 128);
        q_voff = lane < (BN + 127) / 128 ? nb * kblocks * 4 : 0x7fffffff;
        q_ld = 4;
      } else {
        const int c = (wave - kQA) * 64 + lane;
        q_voff = (c < last_n ? c : last_n) * 4;
        q_ld = (int)g.sb_ld * 4;
        q_base = (int)n0 * 4;
      }
    }
    q_dst = uniform(q_dst);
    q_ld = uniform(q_ld);
    q_base = uniform(q_base);
  };
  scale_offsets();
  // LDS destination of this wave's instruction: stage st's scale vectors
  uint8_t* const q_to = wave < kQ ? scale_lds + q_dst : dummy_lds + wave_all * 256;
  const int q_stride = uniform(wave < kQ ? kScaleStage : 0);
  auto load_scales = [&](int kt, int st) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_q, (lds_void*)(q_to + st * q_stride), 4, q_voff,
                                             q_base + kt * q_ld, 0, 0);
  };

  const TileLoader<BM, kWaves> ldA(g.A, g.lda, m0, g.M, wave);
  const TileLoader<BN, kWaves> ldB(g.B, g.ldb, n0, g.N, wave);
  // prologue: stages 0 .. kStages - 2 (each wave issues kSlots loads per
  // stage, with the scale slot first)
  auto prologue = [&]() {
    if constexpr (kStages == 2) {
      // stage 0, then stage 1's B tile (see the schedule below)
      if constexpr (kBlockScaled) load_scales(kb(0), 0);
      ldA.load(kb(0) * kBK, lds, wave);
      ldB.load(kb(0) * kBK, lds + kTileA, wave);
      if (KT > 1) ldB.load(kb(1) * kBK, lds + kStage + kTileA, wave);
    } else {
      for (int st = 0; st < kStages - 1 && st < KT; ++st) {
        if constexpr (kBlockScaled) load_scales(kb(st), st);
        ldA.load(kb(st) * kBK, lds + st * kStage, wave);
        ldB.load(kb(st) * kBK, lds + st * kStage + kTileA, wave);
      }
    }
  };
  prologue();

  // a VALU result computed from the last MFMA output of the previous step
  float done = 0.0f;
  // The vector-memory work of a step (the loads of stage kt+1) is a list of
  // kSlots direct-to-LDS instructions per wave: its scale-vector load (for
  // the blockwise pairs; waves past kQ have none), its A row groups, its B
  // row groups.  They go out two or three at a time,
  // between the matrix instructions: issued all at once they would stall the
  // wave on the vector-memory queue, which drains at about 64 bytes per clock
  // per CU.
  constexpr int kPerA = TileLoader<BM, kWaves>::kPerWave, kPerB = TileLoader<BN, kWaves>::kPerWave;
  constexpr int kS0 = kBlockScaled ? 1 : 0;
  constexpr int kSlots = kS0 + kPerA + kPerB;
  // kPre slots go out right after the barrier, while the wave waits for its
  // first fragments; the rest kPerStrip per strip
  constexpr int kPre = TI >= 8 ? 2 : 0;
  constexpr int kPerStrip = (kSlots - kPre + TI - 1) / TI > 2 ? (kSlots - kPre + TI - 1) / TI : 2;
  // With two stages the B tile is loaded two steps ahead.  A wave reads its
  // B fragments at the start of a step, so after a second barrier (once
  // every wave holds them, after the first strip's MFMAs) the B half of the
  // current stage is free: the next-but-one stage's B tile goes there during
  // the second half of the step, while the next stage's scales and A tile go
  // out in the first half.  The post-barrier burst halves and the B loads
  // get one and a half steps to land.
  constexpr bool kSplitB = kStages == 2;
  constexpr int kNA = kS0 + kPerA;                                   // A-part slots
  constexpr int kPerStripA = (kNA - kPre + TI / 2 - 1) / (TI / 2) > 1 ? (kNA - kPre + TI / 2 - 1) / (TI / 2) : 1;
  constexpr int kPerStripB = (kPerB + TI / 2 - 1) / (TI / 2);        // strips TI/2 .. TI-1
  static_assert(kQ <= kWaves, "at most one scale-vector load per wave and step");
  // LDS reads of the step's scales, issued after the first strip's MFMAs
  constexpr int kScaleReads = PAIR == kPairBlock ? TI + 1 : (PAIR == kPairBlockK ? TI + TJ : 0);
  static_assert(kScaleReads + 2 <= 15, "outstanding LDS reads must fit the lgkm counter");

  // One K step; kMore: the loads of stage kt + kStages - 1 go out during
  // it (all but the last kStages - 1 steps, which run without, so that no
  // step carries a branch).
  // kMore: with two stages, the next stage's A tile and scales go out
  // (kMoreB: and the next-but-one's B tile); with more stages, all loads
  // of stage kt + kStages - 1.
  auto step = [&](const int kt, auto more_c, auto more_b_c) __attribute__((always_inline)) {
    constexpr bool kMore = decltype(more_c)::value;
    constexpr bool kMoreB = decltype(more_b_c)::value;
    const int cur_st = kt % kStages, nxt_st = (kt + kStages - 1) % kStages;
    uint8_t* cur = lds + cur_st * kStage;
    uint8_t* cur_scales = scale_lds + cur_st * kScaleStage;
    uint8_t* nxt = lds + nxt_st * kStage;
    const int k_nxt = kb(kt + kStages - 1) * kBK;
    const int k_b2 = kb(kt + 2 < KT ? kt + 2 : KT - 1) * kBK;  // two-stage B tile
    // this wave's loads of stage kt have landed: only those of later stages
    // may still be in flight (two stages: stage kt+1's B tile, issued last)
    if constexpr (kSplitB) {
      if constexpr (kMore)
        wait_vmem<kPerB>();
      else
        wait_vmem<0>();
    } else {
      if constexpr (kMore)
        wait_vmem<(kStages - 2) * kSlots>();
      else
        wait_vmem<0>();
    }
    // Tile kt and its scales are in LDS for every wave (each waited for its
    // own loads) and the stage the loads of this step overwrite, kt - 1's,
    // is free (each wave waited for its LDS reads before using them).  A
    // bare barrier: __syncthreads() would add a release fence waiting for
    // every load in flight.
    asm volatile("s_barrier" ::: "memory");
    // Vector-memory slot Q of strip I (I = -1: the ones right after the
    // barrier).  Within a strip each goes out right after one of the
    // strip's MFMAs, so a stall on the queue overlaps that MFMA.
    auto issue_slot = [&](auto sc, auto kb_c) {  // slot S; kb_c: B tile two stages ahead
      constexpr int S = decltype(sc)::value;
      if constexpr (S < kS0)
        load_scales(kb(kt + kStages - 1), nxt_st);
      else if constexpr (S - kS0 < kPerA)
        ldA.template load_group<(S - kS0 < kPerA ? S - kS0 : 0)>(k_nxt, nxt, wave);
      else if constexpr (decltype(kb_c)::value)
        ldB.template load_group<(S - kS0 >= kPerA ? S - kS0 - kPerA : 0)>(k_b2, cur + kTileA, wave);
      else
        ldB.template load_group<(S - kS0 >= kPerA ? S - kS0 - kPerA : 0)>(k_nxt, nxt + kTileA, wave);
    };
    constexpr int kQMax = kSplitB ? (kPre > kPerStripA + kPerStripB ? kPre : kPerStripA + kPerStripB)
                                  : (kPre > kPerStrip ? kPre : kPerStrip);
    auto issue_one = [&](auto ic, auto qc) {
      constexpr int I = decltype(ic)::value, Q = decltype(qc)::value;
      if constexpr (kSplitB) {
        // A part: kPre after the barrier, then kPerStripA per strip; B part:
        // kPerStripB per strip from strip TI/2 on
        constexpr int SA = I < 0 ? Q : kPre + I * kPerStripA + Q;
        constexpr bool a_here = (I < 0 ? Q < kPre : Q < kPerStripA) && SA < kNA;
        constexpr int QB = I < 0 ? -1 : (SA < kNA ? Q - kPerStripA : Q - kPerStripA);
        constexpr int SB = kNA + (I - TI / 2) * kPerStripB + QB;
        constexpr bool b_here = I >= TI / 2 && QB >= 0 && QB < kPerStripB && SB < kSlots;
        if constexpr (kMore && a_here) issue_slot(std::integral_constant<int, SA>{}, std::false_type{});
        if constexpr (kMoreB && b_here) issue_slot(std::integral_constant<int, SB>{}, std::true_type{});
      } else {
        constexpr int S = I < 0 ? Q : kPre + I * kPerStrip + Q;
        if constexpr (kMore && S < kSlots && (I < 0 ? Q < kPre : Q < kPerStrip))
          issue_slot(std::integral_constant<int, S>{}, std::false_type{});
      }
    };
    auto issue_strip = [&](auto ic) {
      static_for<kQMax>([&](auto qc) { issue_one(ic, qc); });
    };
    // the second barrier of a two-stage step (after the first strip's
    // MFMAs: every wave holds its B fragments)
    auto mid_barrier = [&]() {
      if constexpr (kSplitB && kMoreB) {
        sched_fence();
        asm volatile("s_barrier" ::: "memory");
        sched_fence();
      }
    };
    // after MFMA j of a strip: its vector-memory slot (after the strip's
    // last MFMA, any slots beyond the strip's MFMA count too)
    auto after_mfma = [&](auto ic, auto jc) {
      constexpr int j = decltype(jc)::value;
      sched_fence();
      issue_one(ic, jc);
      if constexpr (j == TJ - 1)
        static_for<(kQMax > TJ ? kQMax - TJ : 0)>(
            [&](auto qc) { issue_one(ic, std::integral_constant<int, TJ + decltype(qc)::value>{}); });
      sched_fence();
    };

    // Fragment reads of the first two strips: A strip 0, the B fragments,
    // A strip 1.  The MFMAs of strip 0 each wait only for their own B
    // fragment.  Every MFMA of the previous step has completed here: its
    // outputs were consumed by VALU work (the promotion FMAs, or the `done`
    // product below), which the reads' addresses depend on.
    const v8i none = {};
    const FragAddr fa = frag_addr(cur + wm * 128), fb = frag_addr(cur + kTileA + wn * 128);
    // power-of-two scales enter strip 0's MFMAs: read its row scale and the
    // weight block's scale before the fragments, so the first fragment wait
    // covers them; the row scales of later strips follow strip by strip
    const uint32_t sa_addr = lds_addr(cur_scales) + (wm + (lane & 15)) * 4;
    float sa_e[TI], sb_e = 0.f;
    if constexpr (PAIR == kPairBlockE8) {
      sb_e = lds_read_f32(lds_addr(cur_scales + kScaleA) + (wn / 128) * 4, 0);
      sa_e[0] = lds_read_f32(sa_addr, 0);
    }
    v8i af = read_frag<0>(fa, none, none, done);
    v8i bf[TJ];
    static_for<TJ>([&](auto j) { bf[j] = read_frag<j * 2048>(fb, none, none, done); });
    v8i af_next = af;
    if constexpr (TI > 1) af_next = read_frag<2048>(fa, none, none, done);
    constexpr int kNextReads = TI > 1 ? 2 : 0;
    issue_strip(std::integral_constant<int, -1>{});
    auto wait_b = [&](auto jc) {  // before strip 0's MFMA with B fragment j
      constexpr int j = decltype(jc)::value;
      if constexpr (j == 0)
        lds_wait2<2 * (TJ - 1) + kNextReads>(af, bf[0]);
      else
        lds_wait<2 * (TJ - 1 - j) + kNextReads>(bf[j]);
    };

    float sa[TI], sb[TJ][4], sb0 = 0.f;
    auto read_scales = [&]() {
      if (kBlockScaled) {
        const uint32_t a_addr = lds_addr(cur_scales) + (wm + (lane & 15)) * 4;
#pragma unroll
        for (int i = 0; i < TI; ++i) sa[i] = lds_read_f32(a_addr, i * 64);
      }
      if (PAIR == kPairBlock) sb0 = lds_read_f32(lds_addr(cur_scales + kScaleA) + (wn / 128) * 4, 0);
      if (PAIR == kPairBlockK) {
        const uint32_t b_addr = lds_addr(cur_scales + kScaleA) + (wn + (lane >> 4) * 4) * 4;
#pragma unroll
        for (int j = 0; j < TJ; ++j) lds_read_f32x4(b_addr + j * 64, sb[j]);
      }
    };
    auto scales_ready = [&]() {  // after an lgkm wait that covers the scale reads
      if (kBlockScaled) {
#pragma unroll
        for (int i = 0; i < TI; ++i) asm volatile("" : "+v"(sa[i]));
      }
      if (PAIR == kPairBlock) asm volatile("" : "+v"(sb0));
      if (PAIR == kPairBlockK) {
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) asm volatile("" : "+v"(sb[j][r]));
      }
    };

    if constexpr (!kPromote) {
      // Whole-K accumulation in the MFMA accumulator.  Strip i multiplies
      // with af; the fragment of strip i+2 is read into registers that are
      // neither af nor af_next (early clobber against them via `busy`) once
      // the MFMAs of strip i-1 are done (their output is multiplied into
      // `done` first), so it never overwrites a source still being read.
      // With power-of-two scales, strip i+1's row scale is read just before
      // that fragment, so the same wait covers it.
      int se_b = 0;
      static_for<TI>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        int se_a = 0;
        static_for<TJ>([&](auto jc) {
          constexpr int j = decltype(jc)::value;
          if constexpr (i == 0) {
            wait_b(jc);
            if constexpr (PAIR == kPairBlockE8 && j == 0) {
              asm volatile("" : "+v"(sb_e), "+v"(sa_e[0]));
              se_b = e8m0_of(sb_e);
            }
          }
          if constexpr (PAIR == kPairBlockE8) {
            if constexpr (j == 0) se_a = e8m0_of(sa_e[i]);
            acc[i][j] = mfma_16x16x128_e8(bf[j], af, acc[i][j], se_b, se_a);
          } else {
            acc[i][j] = mfma_16x16x128<FMT>(bf[j], af, acc[i][j]);
          }
          after_mfma(ic, jc);
        });
        if constexpr (i == 0) mid_barrier();
        if constexpr (PAIR == kPairBlockE8 && i + 1 < TI) sa_e[i + 1] = lds_read_f32(sa_addr, (i + 1) * 64);
        v8i af_after = af_next;
        if constexpr (i + 2 < TI) {
          if constexpr (i > 0) done = acc[i - 1][TJ - 1][3] * 0.0f;
          af_after = read_frag<(i + 2) * 2048>(fa, af, af_next, done);
          lds_wait<2>(af_next);  // af_next ready; af_after may be in flight
        } else if constexpr (i + 1 < TI) {
          lds_wait<0>(af_next);  // the last fragment
        }
        if constexpr (PAIR == kPairBlockE8 && i + 1 < TI) asm volatile("" : "+v"(sa_e[i + 1]));
        af = af_next;
        af_next = af_after;
      });
      done = acc[TI - 1][TJ - 1][3] * 0.0f;
    } else {
      // Row strips of the wave tile, software pipelined: the MFMAs of strip
      // i+1 (into zeroed partials) are issued before the FMAs that fold the
      // scaled partials of strip i into the accumulators.  Three A fragments
      // rotate: af (strip i, its MFMAs possibly still in flight), af_next
      // (strip i+1), and the one read at the top of strip i for strip i+2,
      // into registers away from both and only after the FMAs of strip i-1
      // consumed the results of its MFMAs (so those are done).  An empty asm
      // makes strip i+1's A fragment depend on the finished accumulators of
      // strip i-1, so the compiler cannot hoist later MFMAs: at most two
      // strips of partials are live, which keeps two waves per SIMD within
      // the register file.
      const v4f zero = {0.f, 0.f, 0.f, 0.f};
      v4f p[TJ], p_next[TJ];
      static_for<TJ>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        wait_b(jc);
        p[j] = mfma_16x16x128<FMT>(bf[j], af, zero);
        sched_fence();
      });
      mid_barrier();
      read_scales();
      static_for<TI>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        constexpr int kAfter = i + 2 < TI ? 2 : 0;  // reads of af_after
        v8i af_after = af_next;
        if constexpr (i + 2 < TI)
          af_after = read_frag<(i + 2) * 2048>(fa, af, af_next, i > 0 ? acc[i > 0 ? i - 1 : 0][TJ - 1][3] : done);
        if constexpr (i + 1 < TI) {
          if constexpr (i > 0) order_after(af_next, acc[i - 1]);
          // af_next was read before the scales (strip 0) or a strip ago
          lds_wait<kAfter + (i == 0 ? kScaleReads : 0)>(af_next);
          static_for<TJ>([&](auto jc) {
            constexpr int j = decltype(jc)::value;
            p_next[j] = mfma_16x16x128<FMT>(bf[j], af_next, zero);
            after_mfma(ic, jc);
          });
        } else {
          sched_fence();
          issue_strip(ic);
          sched_fence();
        }
        if constexpr (i == 0) {
          asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(kAfter));
          scales_ready();
        }
        const float si = PAIR == kPairBlock ? sa[i] * sb0 : sa[i];
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            if (PAIR == kPairBlock)
              acc[i][j][r] = __builtin_fmaf(p[j][r], si, acc[i][j][r]);
            else
              acc[i][j][r] = __builtin_fmaf(p[j][r] * si, sb[j][r], acc[i][j][r]);
          }
        }
#pragma unroll
        for (int j = 0; j < TJ; ++j) p[j] = p_next[j];
        af = af_next;
        af_next = af_after;
      });
      done = acc[TI - 1][TJ - 1][3];
    }
  };
  auto all_steps = [&]() {
    int kt = 0;
    if constexpr (kSplitB) {
      // (the B load of step KT-2 re-reads stage KT-1's B tile into a buffer
      // nothing reads again: a third copy of the step body, without it,
      // would push the kernel past its registers)
      for (; kt + 1 < KT; ++kt) step(kt, std::true_type{}, std::true_type{});
      step(kt, std::false_type{}, std::false_type{});
    } else {
      for (; kt + kStages - 1 < KT; ++kt) step(kt, std::true_type{}, std::false_type{});
      for (; kt < KT; ++kt) step(kt, std::false_type{}, std::false_type{});
    }
  };

  all_steps();

  if constexpr (KS > 1) {
    // the groups' partial tiles: group k > 0 writes its accumulators to LDS
    // (the operand stages are free once every load has landed and every
    // wave is past its last step), group 0 adds them in group order
    float* const red = reinterpret_cast<float*>(lds_all);
    static_assert((KS - 1) * kWaves * TI * TJ * 4 * 64 * 4 <= KS * kGroupBytes, "partials fit the stages");
    wait_vmem_all();
    __syncthreads();
    if (kg > 0) {
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            red[(((kg - 1) * kWaves + wave) * (TI * TJ * 4) + (i * TJ + j) * 4 + r) * 64 + lane] = acc[i][j][r];
    }
    __syncthreads();
    if (kg == 0) {
#pragma unroll
      for (int k = 1; k < KS; ++k)
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int j = 0; j < TJ; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              acc[i][j][r] += red[(((k - 1) * kWaves + wave) * (TI * TJ * 4) + (i * TJ + j) * 4 + r) * 64 + lane];
    }
  }

  if constexpr (SPLITK) {
    static_assert(KS == 1 && !QOUT, "split-K: one group, bf16 output");
    if (!splitk_reduce<TI, TJ, BM * BN>(g, acc, split, tile, wave, lane, dummy_lds)) return;
  }

  // Epilogue: whole-K scales for tensor / row pairs, bf16 RNE, then the
  // tile goes through LDS (the operand stages are free now) so that global
  // stores are whole 16-byte chunks of contiguous C rows.  LDS row m of the
  // tile holds BN bf16; its 16-byte chunk c sits at chunk c ^ (m & 15), which
  // keeps both the 8-byte writes (16 rows, same columns) and the 16-byte
  // reads (one row) free of bank conflicts.
  // The rounding runs before the barrier, so that it overlaps the wait for
  // the slowest wave and the last MFMAs.
  static_assert(BM * BN * 2 <= kStages * kStage, "C tile must fit in the LDS stages");
  const int voff_m = (lane & 15) * 4, voff_n = (lane >> 4) * 16;
  float st = 1.0f;
  if (PAIR == kPairTensor) st = load_f32(rsA, 0, 0) * load_f32(rsB, 0, 0);
  uint2 packed[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    const float sm = PAIR == kPairRow ? load_f32(rsA, voff_m + i * 64, mw * 4) : 1.0f;
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        v[r] = acc[i][j][r];
        if (PAIR == kPairTensor) v[r] = v[r] * st;
        if (PAIR == kPairRow) v[r] = (v[r] * sm) * load_f32(rsB, voff_n + j * 64 + r * 4, nw * 4);
      }
      packed[i][j] = make_uint2(bf16x2_rne(v[0], v[1]), bf16x2_rne(v[2], v[3]));
    }
  }
  wait_vmem_all();  // no load may still be writing LDS
  __syncthreads();  // every wave is done with the operand stages (and the partials)
  constexpr int kRowBytes = BN * 2;
  constexpr int kChunkMask = kRowBytes / 16 < 16 ? kRowBytes / 16 - 1 : 15;  // the swizzle stays in the row
  if (kg == 0) {
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      const int mt = wm + i * 16 + (lane & 15);  // row within the tile
#pragma unroll
      for (int j = 0; j < TJ; ++j) {
        const int nt = wn + j * 16 + (lane >> 4) * 4;  // column within the tile
        const int chunk = (nt * 2) >> 4, half = ((nt * 2) >> 3) & 1;
        *reinterpret_cast<uint2*>(lds_all + mt * kRowBytes + ((chunk ^ (mt & kChunkMask)) << 4) + half * 8) =
            packed[i][j];
      }
    }
  }
  __syncthreads();
  constexpr int kChunksPerRow = kRowBytes / 16;
  constexpr int kThreads = KS * kWaves * 64;
  constexpr int kRowsPerPass = kThreads / kChunksPerRow;
  if constexpr (QOUT) {
    static_assert(kChunksPerRow % 16 == 0, "a 128-column unit per DPP row");
    store_quantized<BM / kRowsPerPass, kRowBytes, kChunkMask, kRowsPerPass>(g, lds_all, m0, n0, kChunksPerRow);
    return;
  }
  const int c = threadIdx.x % kChunksPerRow;
  const int64_t n = n0 + c * 8;
#pragma unroll 4
  for (int mt = threadIdx.x / kChunksPerRow; mt < BM; mt += kRowsPerPass) {
    const int64_t m = m0 + mt;
    if (m >= g.M || n >= g.N) continue;
    const uint4 v = *reinterpret_cast<const uint4*>(lds_all + mt * kRowBytes + ((c ^ (mt & kChunkMask)) << 4));
    uint16_t* dst = g.C + m * g.ldc + n;
    if (n + 8 <= g.N) {
      // non-temporal: C is not read again here, and streaming it out keeps
      // the last-level cache clean for the operands and for the kernels
      // that follow (its write-back then overlaps this compute-bound kernel)
      if (g.c_aligned16) {
        const v4u vv = {v.x, v.y, v.z, v.w};
        __builtin_nontemporal_store(vv, reinterpret_cast<v4u*>(dst));
      } else {
        const v2u lo = {v.x, v.y}, hi = {v.z, v.w};
        __builtin_nontemporal_store(lo, reinterpret_cast<v2u*>(dst));
        __builtin_nontemporal_store(hi, reinterpret_cast<v2u*>(dst) + 1);
      }
    } else {
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
      for (int e = 0; n + e < g.N; ++e) dst[e] = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
    }
  }
}

template <int PAIR, int BM, int BN, int WM, int WN, bool QOUT, int FMT, int KS = 1>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64 * KS) void gemm_kernel(GemmArgs g) {
  int tm, tn;
  tile_coords<BM, BN>(g.M, g.N, g.K, blockIdx.x, tm, tn);
  gemm_tile<PAIR, BM, BN, WM, WN, QOUT, FMT, KS>(g, tm, tn);
}

// Split-K: g.splits workgroups per 128 x 128 tile.  Positions run split by
// split over the tile raster, so the tiles of one split (which share the A
// rows of its K range) sit on neighbouring XCDs, and the two tile rows of
// a 256-row problem that share B rows on one XCD.
template <int PAIR, int BM, int BN, int WM, int WN, int FMT>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64) void gemm_splitk_kernel(GemmArgs g) {
  const int tiles = (int)((g.M + BM - 1) / BM) * (int)((g.N + BN - 1) / BN);
  const int id = xcd_order(tiles * g.splits, blockIdx.x);
  const int split = id / tiles, t = id - split * tiles;
  int tm, tn;
  raster<BM, BN>(g.M, g.N, g.K, t, tm, tn);
  gemm_tile<PAIR, BM, BN, WM, WN, false, FMT, 1, true>(g, tm, tn, split, t);
}

// Grouped GEMM: one launch over several problems that share the pair, the
// formats and K (the fused QKV or gate / up projections: one activation
// operand, several weights and outputs).  The workgroups' XCD-ordered
// positions run over the problems' rasters one after another; the problem
// of a position is found from the prefix sums of the tile counts.
template <int PAIR, int BM, int BN, int WM, int WN, int KS = 1>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64 * KS) void gemm_grouped_kernel(GemmGroup gs) {
  const int id = xcd_order(gs.tile_start[gs.count], blockIdx.x);
  int p = 0;
  for (int i = 1; i < gs.count; ++i) p += id >= gs.tile_start[i] ? 1 : 0;
  int tm, tn;
  raster<BM, BN>(gs.prob[p].M, gs.prob[p].N, gs.prob[p].K, id - gs.tile_start[p], tm, tn);
  gemm_tile<PAIR, BM, BN, WM, WN, false, 0, KS>(gs.prob[p], tm, tn);
}

template <int PAIR, int BM, int BN, int WM, int WN, bool QOUT, int FMT, int KS = 1>
hipError_t launch_tiles(const GemmArgs& g, hipStream_t s) {
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  if (tiles <= 0 || tiles > 0x7fffffff) return hipErrorInvalidValue;
  constexpr int threads = (BM / WM) * (BN / WN) * 64 * KS;
  gemm_kernel<PAIR, BM, BN, WM, WN, QOUT, FMT, KS><<<dim3((unsigned)tiles), threads, 0, s>>>(g);
  return hipGetLastError();
}

// Two K groups per 64 x 64 tile (one workgroup of 8 waves per CU) when there
// are at most 256 such tiles, so that a CU would hold one workgroup anyway,
// and the K blocks split evenly; more tiles keep two 4-wave workgroups per
// CU (measured: 256 x 12288 x 4096 35 -> 28 us with groups, 256 x 4096 x
// 12288 with its 768 tiles 31 -> 34 us).
inline bool k_groups(const GemmArgs& g) {
  return ((g.M + 63) / 64) * ((g.N + 63) / 64) <= 256 && (g.K / kBK) % 2 == 0;
}

// 256 x 256 tiles (8 waves of 128 x 64) when they fill the chip at least
// twice over; else 128 x 128 tiles (4 waves of 64 x 64) when they fill it
// once; else, for skinny problems such as a decode step, whose time goes
// into streaming the weights: 64 x 64 tiles with two K groups when those
// fit (k_groups), 128 x 128 tiles of 8 waves of 32 x 64 with a four-stage
// ring (one workgroup per CU) when there are 128 to 255 of them, and 64 x 64
// tiles (4 waves of 32 x 32) below that.  Every choice but the K groups sums
// an output's K blocks in the same order.  Quantized output needs whole
// 128-column units in a tile: 256 or 128 tiles only.
template <int PAIR, bool QOUT, int FMT>
hipError_t launch_pair(const GemmArgs& g, hipStream_t s) {
  const int64_t big_tiles = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  const int64_t mid_tiles = ((g.M + 127) / 128) * ((g.N + 127) / 128);
  if constexpr (PAIR != kPairBlockK) {
    if (big_tiles >= 512) return launch_tiles<PAIR, 256, 256, 128, 64, QOUT, FMT>(g, s);
  }
  if constexpr (QOUT) {
    return launch_tiles<PAIR, 128, 128, 64, 64, QOUT, FMT>(g, s);
  } else {
    if (mid_tiles >= 256) return launch_tiles<PAIR, 128, 128, 64, 64, QOUT, FMT>(g, s);
    if (k_groups(g)) return launch_tiles<PAIR, 64, 64, 32, 32, QOUT, FMT, 2>(g, s);
    if (mid_tiles >= 128) return launch_tiles<PAIR, 128, 128, 32, 64, QOUT, FMT>(g, s);
    return launch_tiles<PAIR, 64, 64, 32, 32, QOUT, FMT>(g, s);
  }
}

// The kernels address operands with 32-bit offsets: split the problem into
// sub-GEMMs whose A and B row ranges each span less than 4 GiB.
template <int PAIR, bool QOUT, int FMT>
hipError_t launch_split(const GemmArgs& g, hipStream_t s) {
  // 32-bit offsets: each sub-problem's A rows, B rows and C rows span
  // < 2 GiB, and row / column indices stay below 2^31 / 4
  const int64_t lim = (int64_t)1 << 31;
  int64_t mstep = g.M, nstep = g.N;
  if (g.M * g.lda >= lim) mstep = ((lim - 1) / g.lda) / 256 * 256;
  const int64_t c_row_bytes = QOUT ? g.ldq : 2 * g.ldc;
  if (g.M * c_row_bytes >= lim) {
    const int64_t cstep = ((lim - 1) / c_row_bytes) / 256 * 256;
    if (cstep < mstep) mstep = cstep;
  }
  // column steps in whole 2048-column pairs of bands, so that a
  // sub-problem's tiles take the K direction of their global columns
  // (odd 1024-column bands walk K backwards)
  if (g.N * g.ldb >= lim) {
    const int64_t q = (lim - 1) / g.ldb;
    nstep = q >= 2048 ? q / 2048 * 2048 : q / 256 * 256;
  }
  if (mstep > ((int64_t)1 << 28)) mstep = (int64_t)1 << 28;
  if (nstep > ((int64_t)1 << 28)) nstep = (int64_t)1 << 28;
  if (mstep <= 0 || nstep <= 0) return hipErrorInvalidValue;
  for (int64_t m = 0; m < g.M; m += mstep) {
    for (int64_t n = 0; n < g.N; n += nstep) {
      GemmArgs sub = g;
      sub.M = (g.M - m) < mstep ? (g.M - m) : mstep;
      sub.N = (g.N - n) < nstep ? (g.N - n) : nstep;
      sub.A = g.A + m * g.lda;
      sub.B = g.B + n * g.ldb;
      if (QOUT) {
        sub.Cq = g.Cq + m * g.ldq + n;
        sub.Cs = g.Cs + (n / 128) * g.cs_ld + m;  // n is a multiple of 256
      } else {
        sub.C = g.C + m * g.ldc + n;
      }
      // scale arrays keep the full problem's layout (strides sa_ld, sb_ld);
      // re-base them at the sub-problem's first row / column
      int64_t da = 0, db = 0;
      if (PAIR != kPairTensor) da = m;
      if (PAIR == kPairRow || PAIR == kPairBlockK) db = n;
      if (PAIR == kPairBlock || PAIR == kPairBlockE8) db = (n / 128) * (g.K / 128);
      sub.sA = g.sA + da;
      sub.sB = g.sB + db;
      sub.sa_count = g.sa_count - da;
      sub.sb_count = g.sb_count - db;
      hipError_t e = launch_pair<PAIR, QOUT, FMT>(sub, s);
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

// Explicit instantiations: the host pass otherwise emits launch stubs only
// for the first instantiated pair.
#define FP8Q_GEMM_KERNEL(PAIR, BM, BN, WM, WN) \
  template __global__ void gemm_kernel<PAIR, BM, BN, WM, WN, false, 0>(GemmArgs);
// the backward pairs with E5M2 operands (formats 1, 2, 3)
#define FP8Q_GEMM_KERNEL_FMT(PAIR, BM, BN, WM, WN)                               \
  template __global__ void gemm_kernel<PAIR, BM, BN, WM, WN, false, 1>(GemmArgs); \
  template __global__ void gemm_kernel<PAIR, BM, BN, WM, WN, false, 2>(GemmArgs); \
  template __global__ void gemm_kernel<PAIR, BM, BN, WM, WN, false, 3>(GemmArgs);
FP8Q_GEMM_KERNEL(kPairTensor, 256, 256, 128, 64)
FP8Q_GEMM_KERNEL(kPairTensor, 128, 128, 64, 64)
FP8Q_GEMM_KERNEL(kPairRow, 256, 256, 128, 64)
FP8Q_GEMM_KERNEL(kPairRow, 128, 128, 64, 64)
FP8Q_GEMM_KERNEL(kPairBlock, 256, 256, 128, 64)
FP8Q_GEMM_KERNEL(kPairBlock, 128, 128, 64, 64)
FP8Q_GEMM_KERNEL(kPairBlockK, 128, 128, 64, 64)
FP8Q_GEMM_KERNEL(kPairTensor, 128, 128, 32, 64)
FP8Q_GEMM_KERNEL(kPairRow, 128, 128, 32, 64)
FP8Q_GEMM_KERNEL(kPairBlock, 128, 128, 32, 64)
FP8Q_GEMM_KERNEL(kPairBlockK, 128, 128, 32, 64)
FP8Q_GEMM_KERNEL(kPairBlockE8, 128, 128, 32, 64)
FP8Q_GEMM_KERNEL(kPairTensor, 64, 64, 32, 32)
FP8Q_GEMM_KERNEL(kPairRow, 64, 64, 32, 32)
FP8Q_GEMM_KERNEL(kPairBlock, 64, 64, 32, 32)
FP8Q_GEMM_KERNEL(kPairBlockK, 64, 64, 32, 32)
FP8Q_GEMM_KERNEL(kPairBlockE8, 256, 256, 128, 64)
FP8Q_GEMM_KERNEL(kPairBlockE8, 128, 128, 64, 64)
FP8Q_GEMM_KERNEL(kPairBlockE8, 64, 64, 32, 32)
FP8Q_GEMM_KERNEL_FMT(kPairBlock, 256, 256, 128, 64)
FP8Q_GEMM_KERNEL_FMT(kPairBlock, 128, 128, 64, 64)
FP8Q_GEMM_KERNEL_FMT(kPairBlock, 128, 128, 32, 64)
FP8Q_GEMM_KERNEL_FMT(kPairBlockK, 128, 128, 32, 64)
FP8Q_GEMM_KERNEL_FMT(kPairBlock, 64, 64, 32, 32)
FP8Q_GEMM_KERNEL_FMT(kPairBlockK, 128, 128, 64, 64)
FP8Q_GEMM_KERNEL_FMT(kPairBlockK, 64, 64, 32, 32)
#undef FP8Q_GEMM_KERNEL
#undef FP8Q_GEMM_KERNEL_FMT
#define FP8Q_GEMM_KERNEL_KS2(PAIR, FMT) template __global__ void gemm_kernel<PAIR, 64, 64, 32, 32, false, FMT, 2>(GemmArgs);
FP8Q_GEMM_KERNEL_KS2(kPairTensor, 0)
FP8Q_GEMM_KERNEL_KS2(kPairRow, 0)
FP8Q_GEMM_KERNEL_KS2(kPairBlockE8, 0)
FP8Q_GEMM_KERNEL_KS2(kPairBlock, 0)
FP8Q_GEMM_KERNEL_KS2(kPairBlock, 1)
FP8Q_GEMM_KERNEL_KS2(kPairBlock, 2)
FP8Q_GEMM_KERNEL_KS2(kPairBlock, 3)
FP8Q_GEMM_KERNEL_KS2(kPairBlockK, 0)
FP8Q_GEMM_KERNEL_KS2(kPairBlockK, 1)
FP8Q_GEMM_KERNEL_KS2(kPairBlockK, 2)
FP8Q_GEMM_KERNEL_KS2(kPairBlockK, 3)
#undef FP8Q_GEMM_KERNEL_KS2
#define FP8Q_GEMM_SPLITK(PAIR) template __global__ void gemm_splitk_kernel<PAIR, 128, 128, 32, 64, 0>(GemmArgs);
FP8Q_GEMM_SPLITK(kPairTensor)
FP8Q_GEMM_SPLITK(kPairRow)
FP8Q_GEMM_SPLITK(kPairBlock)
FP8Q_GEMM_SPLITK(kPairBlockK)
#undef FP8Q_GEMM_SPLITK
template __global__ void gemm_kernel<kPairBlock, 256, 256, 128, 64, true, 0>(GemmArgs);
template __global__ void gemm_kernel<kPairBlock, 128, 128, 64, 64, true, 0>(GemmArgs);
#define FP8Q_GEMM_GROUPED(PAIR)                                                     \
  template __global__ void gemm_grouped_kernel<PAIR, 256, 256, 128, 64>(GemmGroup);    \
  template __global__ void gemm_grouped_kernel<PAIR, 128, 128, 64, 64>(GemmGroup);     \
  template __global__ void gemm_grouped_kernel<PAIR, 64, 64, 32, 32>(GemmGroup);       \
  template __global__ void gemm_grouped_kernel<PAIR, 64, 64, 32, 32, 2>(GemmGroup);
FP8Q_GEMM_GROUPED(kPairTensor)
FP8Q_GEMM_GROUPED(kPairRow)
FP8Q_GEMM_GROUPED(kPairBlock)
#undef FP8Q_GEMM_GROUPED

template <int PAIR, int BM, int BN, int WM, int WN, int KS = 1>
hipError_t launch_grouped_tiles(GemmGroup gs, hipStream_t s) {
  int64_t total = 0;
  for (int i = 0; i < gs.count; ++i) {
    gs.tile_start[i] = (int)total;
    total += ((gs.prob[i].M + BM - 1) / BM) * ((gs.prob[i].N + BN - 1) / BN);
    if (total > 0x7fffffff) return hipErrorInvalidValue;
  }
  gs.tile_start[gs.count] = (int)total;
  if (total <= 0) return hipErrorInvalidValue;
  constexpr int threads = (BM / WM) * (BN / WN) * 64 * KS;
  gemm_grouped_kernel<PAIR, BM, BN, WM, WN, KS><<<dim3((unsigned)total), threads, 0, s>>>(gs);
  return hipGetLastError();
}

// Each problem goes to the kernel a single call would give it.  The tiled
// kernels without K groups all sum K in one order, so one launch takes every
// problem a single call would give one of them (the tile size from their
// tile count over all, as launch_pair chooses it for one: for a skinny
// problem among large ones that is a larger tile than its own, with the same
// bits); the problems a single call would split into K groups (another
// order of the K sum) go to a second launch.
template <int PAIR>
hipError_t launch_grouped_pair(const GemmGroup& gs, hipStream_t s) {
  GemmGroup tiled{}, thin{};
  int64_t big = 0, mid = 0;
  for (int i = 0; i < gs.count; ++i) {
    const GemmArgs& g = gs.prob[i];
    const int64_t big_i = ((g.M + 255) / 256) * ((g.N + 255) / 256);
    const int64_t mid_i = ((g.M + 127) / 128) * ((g.N + 127) / 128);
    if (big_i < 512 && mid_i < 256 && k_groups(g)) {
      thin.prob[thin.count++] = g;
    } else {
      tiled.prob[tiled.count++] = g;
      big += big_i;
      mid += mid_i;
    }
  }
  if (tiled.count) {
    const hipError_t e = big >= 512   ? launch_grouped_tiles<PAIR, 256, 256, 128, 64>(tiled, s)
                         : mid >= 256 ? launch_grouped_tiles<PAIR, 128, 128, 64, 64>(tiled, s)
                                      : launch_grouped_tiles<PAIR, 64, 64, 32, 32>(tiled, s);
    if (e != hipSuccess) return e;
  }
  if (thin.count) return launch_grouped_tiles<PAIR, 64, 64, 32, 32, 2>(thin, s);
  return hipSuccess;
}

}  // namespace gemm_detail

using namespace gemm_detail;

template <int PAIR>
hipError_t launch_formats(const GemmArgs& g, int formats, hipStream_t s) {
  switch (formats) {
    case 0: return launch_split<PAIR, false, 0>(g, s);
    case 1: return launch_split<PAIR, false, 1>(g, s);
    case 2: return launch_split<PAIR, false, 2>(g, s);
    case 3: return launch_split<PAIR, false, 3>(g, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm(const GemmArgs& g, int pair, int formats, hipStream_t s) {
  if (formats != 0 && pair != kPairBlock && pair != kPairBlockK) return hipErrorInvalidValue;
  switch (pair) {
    case kPairTensor: return launch_split<kPairTensor, false, 0>(g, s);
    case kPairRow: return launch_split<kPairRow, false, 0>(g, s);
    case kPairBlock: return launch_formats<kPairBlock>(g, formats, s);
    case kPairBlockK: return launch_formats<kPairBlockK>(g, formats, s);
    case kPairBlockE8: return launch_split<kPairBlockE8, false, 0>(g, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_grouped(const GemmGroup& gs, int pair, hipStream_t s) {
  if (gs.count < 1 || gs.count > kMaxGroup) return hipErrorInvalidValue;
  // 32-bit operand offsets inside the kernel: each problem's A, B and C
  // rows span less than 2 GiB
  const int64_t lim = (int64_t)1 << 31;
  for (int i = 0; i < gs.count; ++i) {
    const GemmArgs& g = gs.prob[i];
    if (g.M * g.lda >= lim || g.N * g.ldb >= lim || g.M * 2 * g.ldc >= lim) return hipErrorInvalidValue;
  }
  switch (pair) {
    case kPairTensor: return launch_grouped_pair<kPairTensor>(gs, s);
    case kPairRow: return launch_grouped_pair<kPairRow>(gs, s);
    case kPairBlock: return launch_grouped_pair<kPairBlock>(gs, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_quantized(const GemmArgs& g, int pair, hipStream_t s) {
  if (pair != kPairBlock || g.N % 128) return hipErrorInvalidValue;
  return launch_split<kPairBlock, true, 0>(g, s);
}

hipError_t launch_gemm_splitk(const GemmArgs& g, int pair, hipStream_t s) {
  if (g.splits <= 1) return launch_gemm(g, pair, 0, s);
  const int64_t tiles = ((g.M + 127) / 128) * ((g.N + 127) / 128);
  if (!g.part || !g.cnt || g.splits > 8 || (g.K / kBK) % g.splits || tiles * g.splits > 256)
    return hipErrorInvalidValue;
  const dim3 grid((unsigned)(tiles * g.splits));
  switch (pair) {
    case kPairTensor: gemm_splitk_kernel<kPairTensor, 128, 128, 32, 64, 0><<<grid, 512, 0, s>>>(g); break;
    case kPairRow: gemm_splitk_kernel<kPairRow, 128, 128, 32, 64, 0><<<grid, 512, 0, s>>>(g); break;
    case kPairBlock: gemm_splitk_kernel<kPairBlock, 128, 128, 32, 64, 0><<<grid, 512, 0, s>>>(g); break;
    case kPairBlockK: gemm_splitk_kernel<kPairBlockK, 128, 128, 32, 64, 0><<<grid, 512, 0, s>>>(g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace fp8q
