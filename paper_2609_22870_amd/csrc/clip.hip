// Calibrated Clipping (paper Sec. 4, Alg. 1, Eq. 5) on gfx950: the new PPO
// clipping bounds of FP8 training from one batch's per-token arrays.
//
// Every statistic the two grid searches need is a sum over tokens, so one
// pass over the batch gathers all of them:
//   * negative-advantage tokens: their count, the count with r_BF16 <=
//     c_low_ref (the reference quantile), the Eq. 5 denominator of the
//     reference ratio (r_BF16 > c_low_ref), and for every lower-grid point
//     L_k the count with r_FP8 <= L_k and the Eq. 5 denominator sum with
//     r_FP8 > L_k;
//   * positive-advantage tokens: their count, the Eq. 5 numerator of the
//     reference ratio (r_BF16 < c_high_ref), and for every upper-grid point
//     H_k the numerator sum with r_FP8 < H_k.
// A token's grid position is found once (an estimate from its ratio,
// corrected by exact comparisons with the float64 grid points) and the
// token is added to that bin of its wave's bins, held in registers (bin r
// in lane r); the threshold sums of every grid point are prefix sums over
// the bins.  Sums are float64 in a fixed order (per thread in token order,
// or per wave in token-group then lane order for the bins, the threads or
// waves of a block in order, the blocks by a fixed lane-then-tree order,
// the bins in order), so the result is the same on every run.  A second
// kernel reduces the blocks and runs the searches and SmoothUpdate.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "fp8q.h"
#include "internal.h"

namespace fp8q {

namespace clip_detail {

// Slots of a block's partial sums (all float64; counts are exact there),
// stored slot-major ([slot][block]): [0] negatives, [1] positives, [2]
// negatives with r_BF16 <= c_low_ref, [3] reference numerator, [4] reference
// denominator, then per lower bin j (the tokens with exactly j lower-grid
// points below r_FP8, j = 0 .. KL) the negative tokens' count and Eq. 5
// denominator sum, then per upper bin j (exactly j upper-grid points at or
// below r_FP8, j = 0 .. KH) the positive tokens' Eq. 5 numerator sum.
template <int KL, int KH>
struct Slots {
  static constexpr int kCount = 5, kDen = kCount + KL + 1, kNum = kDen + KL + 1, kTotal = kNum + KH + 1;
};

// Grid point lo + k * step, rounded once after the product and once after
// the sum (the build does not contract them).
__device__ __forceinline__ double grid_point(double lo, double step, int k) { return (double)k * step + lo; }

// Number of grid points lo + k step (k < n) strictly below r (strict =
// true) or at most r (strict = false).
__device__ __forceinline__ int grid_rank(double r, double lo, double step, double inv_step, int n, bool strict) {
  // (fmin / fmax keep the conversion defined for any input; ratios are
  // finite by contract)
  const double e = fmax(fmin(floor((r - lo) * inv_step) + 1.0, (double)n), 0.0);
  int j = (int)e;
  // the estimate is within one point of the rank (the float64 product
  // differs from the exact quotient by a few units in the last place, far
  // less than a step); settle it exactly with one check each way
  {
    const double g = grid_point(lo, step, j - 1);
    const bool below = strict ? (g < r) : (g <= r);
    j -= (j > 0 && !below) ? 1 : 0;
  }
  {
    const double g = grid_point(lo, step, j);
    const bool below = strict ? (g < r) : (g <= r);
    j += (j < n && below) ? 1 : 0;
  }
  return j;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t o = __shfl_xor(v, off, 64);
    v = o < v ? o : v;
  }
  return v;
}

__device__ __forceinline__ double wave_sum(double v) {
  // fixed butterfly: the same partner order on every run
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Bins of a wave, in registers: val bin r (the lower bins' Eq. 5 denominator
// sums, r = j <= KL, then the upper bins' numerator sums, r = KL + 1 + j) in
// lane r of `lo` (r < 64) or lane r - 64 of `hi`; the lower bins' counts in
// lane j of `cnt`.  A token that falls in one of them (a ratio inside a
// search interval: about one token in a hundred) is added by the bin's
// lane, the wave's binned tokens one after another in lane order, so every
// bin sums in a fixed order and no LDS is needed: the kernel runs three
// waves per SIMD instead of the one that per-thread LDS bins allowed.
template <int KL, int KH>
struct WaveBins {
  static constexpr int kVal = KL + KH + 2, kNum0 = KL + 1;
  static_assert(KL + 1 <= 64 && kVal <= 128, "bins fit two lane sets");
  double lo = 0.0, hi = 0.0;
  int cnt = 0;
};

// Per-thread sums in registers.  Most ratios lie between the two search
// intervals (above the last lower point, below the first upper point), so
// a negative token usually falls in the top lower bin (nl) and a positive
// one in the bottom upper bin (0): those two bins are kept here, per
// thread in token order, and only the other tokens go to the wave's bins.
// A bin is fed by one of the two only.
struct Scalars {
  int n_neg, n_pos, cnt_ref, top_cnt;
  double num_ref, den_ref, top_den, bottom_num;
};

__device__ __forceinline__ double readlane_f64(double v, int l) {
  const uint64_t u = __double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)u, l), hi = __builtin_amdgcn_readlane((uint32_t)(u >> 32), l);
  return __longlong_as_double(((uint64_t)hi << 32) | lo);
}

// l_last: the last lower grid point; a negative token above it has every
// lower point strictly below its ratio (bin nl).  The first upper point is
// h_min; a positive token below it has no upper point at or below its
// ratio (bin 0).
// The token's sums (a token with a = 0, also the padding past the end of a
// range, enters none).  NEG / POS: its sign when the whole wave shares it
// (the tokens of a response share one advantage, and a wave covers 256
// consecutive tokens), which drops the other sign's selects; else both are
// 0 and the token's own sign decides.  Called by every lane of the wave.
template <int KL, int KH, bool NEG, bool POS>
__device__ __forceinline__ void add_token(const ClipArgs& p, double l_last, float a, float w, float pi, float rb,
                                          float rf, Scalars& s, WaveBins<KL, KH>& b) {
  using B = WaveBins<KL, KH>;
  const double rb64 = rb, rf64 = rf;
  const bool neg = NEG || (!POS && a < 0.0f), pos = POS || (!NEG && a > 0.0f);
  const double wp = (double)w * (double)pi;
  const double tb = (wp * rb64) * (double)a, tf = (wp * rf64) * (double)a;
  bool top = false, bottom = false;
  if (!POS) {
    s.n_neg += neg ? 1 : 0;
    s.cnt_ref += (neg && rb64 <= p.c_low_ref) ? 1 : 0;
    s.den_ref += (neg && rb64 > p.c_low_ref) ? tb : 0.0;
    top = neg && rf64 > l_last;
    s.top_cnt += top ? 1 : 0;
    s.top_den += top ? tf : 0.0;
  }
  if (!NEG) {
    s.n_pos += pos ? 1 : 0;
    s.num_ref += (pos && rb64 < p.c_high_ref) ? tb : 0.0;
    bottom = pos && rf64 < p.h_min;
    s.bottom_num += bottom ? tf : 0.0;
  }
  const bool binned = (neg && !top) || (pos && !bottom);
  uint64_t m = __ballot(binned);
  if (m == 0) return;
  // lower bins count the grid points strictly below r_FP8; upper bins the
  // points at or below it
  const int j = binned ? grid_rank(rf64, neg ? p.l_min : p.h_min, p.step, p.inv_step, neg ? p.nl : p.nh, neg) : 0;
  const int row = neg ? j : B::kNum0 + j;
  const int lane = threadIdx.x & 63;
  while (m) {
    const int l = __builtin_ctzll(m);
    m &= m - 1;
    const int r = __builtin_amdgcn_readlane(row, l);
    const double v = readlane_f64(tf, l);
    const bool is_neg = __builtin_amdgcn_readlane(neg ? 1 : 0, l) != 0;
    if (r < 64) {
      b.lo += lane == r ? v : 0.0;
    } else {
      b.hi += lane == r - 64 ? v : 0.0;
    }
    b.cnt += (is_neg && lane == r) ? 1 : 0;
  }
}

// Four consecutive tokens of the five inputs.
struct Group {
  float4 a, w, pi, rb, rf;
};

// The group at token i; tokens at or past `end` read as a = 0 (they enter
// no sum).
__device__ __forceinline__ Group load_group(const ClipArgs& p, int64_t i, int64_t end) {
  Group g;
  if (i + 4 <= end) {
    g.a = *reinterpret_cast<const float4*>(p.adv + i);
    g.w = *reinterpret_cast<const float4*>(p.w + i);
    g.pi = *reinterpret_cast<const float4*>(p.pi + i);
    g.rb = *reinterpret_cast<const float4*>(p.rb + i);
    g.rf = *reinterpret_cast<const float4*>(p.rf + i);
  } else {
    float v[5][4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool ok = i + e < end;
      v[0][e] = ok ? p.adv[i + e] : 0.0f;
      v[1][e] = ok ? p.w[i + e] : 0.0f;
      v[2][e] = ok ? p.pi[i + e] : 0.0f;
      v[3][e] = ok ? p.rb[i + e] : 1.0f;
      v[4][e] = ok ? p.rf[i + e] : 1.0f;
    }
    g.a = make_float4(v[0][0], v[0][1], v[0][2], v[0][3]);
    g.w = make_float4(v[1][0], v[1][1], v[1][2], v[1][3]);
    g.pi = make_float4(v[2][0], v[2][1], v[2][2], v[2][3]);
    g.rb = make_float4(v[3][0], v[3][1], v[3][2], v[3][3]);
    g.rf = make_float4(v[4][0], v[4][1], v[4][2], v[4][3]);
  }
  return g;
}

template <int KL, int KH, bool NEG, bool POS>
__device__ __forceinline__ void add_full_group(const ClipArgs& p, double l_last, const Group& g, Scalars& s,
                                               WaveBins<KL, KH>& b) {
  add_token<KL, KH, NEG, POS>(p, l_last, g.a.x, g.w.x, g.pi.x, g.rb.x, g.rf.x, s, b);
  add_token<KL, KH, NEG, POS>(p, l_last, g.a.y, g.w.y, g.pi.y, g.rb.y, g.rf.y, s, b);
  add_token<KL, KH, NEG, POS>(p, l_last, g.a.z, g.w.z, g.pi.z, g.rb.z, g.rf.z, s, b);
  add_token<KL, KH, NEG, POS>(p, l_last, g.a.w, g.w.w, g.pi.w, g.rb.w, g.rf.w, s, b);
}

// One group per lane, every lane of the wave (wave-uniform branches only).
template <int KL, int KH>
__device__ __forceinline__ void add_group(const ClipArgs& p, double l_last, const Group& g, Scalars& s,
                                          WaveBins<KL, KH>& b) {
  const bool all_neg = g.a.x < 0.f && g.a.y < 0.f && g.a.z < 0.f && g.a.w < 0.f;
  const bool all_pos = g.a.x > 0.f && g.a.y > 0.f && g.a.z > 0.f && g.a.w > 0.f;
  if (__all(all_neg))
    add_full_group<KL, KH, true, false>(p, l_last, g, s, b);
  else if (__all(all_pos))
    add_full_group<KL, KH, false, true>(p, l_last, g, s, b);
  else
    add_full_group<KL, KH, false, false>(p, l_last, g, s, b);
}

// Partial sums of one block's contiguous token range [b * chunk, ...):
// thread t takes the 4-token groups t, t + T, ... of the range, in order,
// with the loads of the next kDepth groups in flight (two: the twelve waves
// of a block already keep enough loads in flight, and deeper staging cost
// registers and time, 51.5 against 46.4 us on the paper's batch).  Every
// lane runs the same number of iterations (groups past the range read as
// a = 0).
template <int KL, int KH, int T>
__global__ __launch_bounds__(T) void clip_stats_kernel(ClipArgs p) {
  using S = Slots<KL, KH>;
  using B = WaveBins<KL, KH>;
  constexpr int kWaves = T / 64;
  __shared__ double red[kWaves][5];
  __shared__ double wval[kWaves][B::kVal];
  __shared__ int wcnt[kWaves][KL + 1];
  Scalars s{0, 0, 0, 0, 0.0, 0.0, 0.0, 0.0};
  WaveBins<KL, KH> bins;
  const double l_last = grid_point(p.l_min, p.step, p.nl - 1);

  constexpr int kDepth = 2;
  constexpr int64_t kStride = 4 * T;
  const int64_t begin = (int64_t)blockIdx.x * p.chunk;
  const int64_t end = begin + p.chunk < p.n ? begin + p.chunk : p.n;
  const int64_t lane0 = 4 * (int64_t)threadIdx.x;
  Group g[kDepth];
#pragma unroll
  for (int d = 0; d < kDepth; ++d) g[d] = load_group(p, begin + lane0 + d * kStride, end);
  for (int64_t base = begin; base < end; base += kDepth * kStride) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      const int64_t id = base + lane0 + d * kStride;
      if (base + d * kStride < end) add_group(p, l_last, g[d], s, bins);  // (uniform)
      g[d] = load_group(p, id + kDepth * kStride, end);
    }
  }

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // the register-held bins (per thread, token order) join the wave's bins
  // (no token was added to those two rows there): wave sums
  const double top_den = wave_sum(s.top_den), bottom_num = wave_sum(s.bottom_num);
  const double top_cnt = wave_sum((double)s.top_cnt);
  // the wave's bins to LDS
  for (int r = lane; r < B::kVal; r += 64) {
    double v = r < 64 ? bins.lo : bins.hi;
    if (r == p.nl) v = top_den;
    if (r == B::kNum0) v = bottom_num;
    wval[wave][r] = v;
  }
  if (lane <= KL) wcnt[wave][lane] = lane == p.nl ? (int)top_cnt : bins.cnt;

  // scalars: wave sums, then the waves in order
  const double sv[5] = {(double)s.n_neg, (double)s.n_pos, (double)s.cnt_ref, s.num_ref, s.den_ref};
#pragma unroll
  for (int q = 0; q < 5; ++q) {
    const double v = wave_sum(sv[q]);
    if (lane == 0) red[wave][q] = v;
  }
  __syncthreads();
  const int64_t out = blockIdx.x;
  if (threadIdx.x < 5) {
    double v = red[0][threadIdx.x];
#pragma unroll
    for (int q = 1; q < kWaves; ++q) v += red[q][threadIdx.x];
    p.partials[(int64_t)threadIdx.x * p.blocks + out] = v;
  }
  // bins: thread r sums row r over the waves, in wave order
  for (int r = threadIdx.x; r < 2 * (KL + 1) + KH + 1; r += T) {
    double v = 0.0;
    int slot;
    if (r < KL + 1) {
      int c = 0;
      for (int w = 0; w < kWaves; ++w) c += wcnt[w][r];
      v = (double)c;
      slot = S::kCount + r;
    } else if (r < 2 * (KL + 1)) {
      const int j = r - (KL + 1);
      for (int w = 0; w < kWaves; ++w) v += wval[w][j];
      slot = S::kDen + j;
    } else {
      const int j = r - 2 * (KL + 1);
      for (int w = 0; w < kWaves; ++w) v += wval[w][B::kNum0 + j];
      slot = S::kNum + j;
    }
    p.partials[(int64_t)slot * p.blocks + out] = v;
  }
}

// Inclusive prefix sums of tot[0 .. n) (n <= 64), lane k getting tot[0] +
// ... + tot[k] summed in index order: the values go to lanes once, then
// one running sum walks them (every lane computes the same sum from
// readlanes) and lane k keeps its prefix.  No lane-dependent loop of LDS
// reads.
__device__ __forceinline__ double prefix_in_order(const double* tot, int n) {
  const int lane = threadIdx.x & 63;
  const double v = lane < n ? tot[lane] : 0.0;
  double run = 0.0, mine = 0.0;
  for (int j = 0; j < n; ++j) {
    run += readlane_f64(v, j);
    mine = lane == j ? run : mine;
  }
  return mine;
}

__device__ __forceinline__ double smooth_update(double b, double b_star, double delta) {
  double d = (b_star - b) / 2.0;
  d = d < -delta ? -delta : d;
  d = d > delta ? delta : d;
  return b + d;
}

// Sums the blocks' partials (slot by slot: lane l takes blocks l, l + 64,
// ... in order, then a fixed shuffle tree), turns the bins into the
// threshold sums of every grid point (in bin order), then Alg. 1's
// searches: L* by matching counts (first minimum), H* by matching the
// Eq. 5 ratio at L* (first minimum), and SmoothUpdate of both bounds.
template <int KL, int KH>
__global__ __launch_bounds__(1024) void clip_search_kernel(ClipArgs p) {
  using S = Slots<KL, KH>;
  constexpr int kPerWave = (S::kTotal + 15) / 16, kPerLane = kClipMaxBlocks / 64;
  __shared__ double tot[S::kTotal];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // every load first (all in flight together), then the sums in order
  double x[kPerWave][kPerLane];
#pragma unroll
  for (int u = 0; u < kPerWave; ++u) {
    const int q = wave + 16 * u;
#pragma unroll
    for (int k = 0; k < kPerLane; ++k) {
      const int b = lane + 64 * k;
      // every lane loads (an in-range element), then keeps it or not
      const int qc = q < S::kTotal ? q : S::kTotal - 1, bc = b < p.blocks ? b : p.blocks - 1;
      const double v = p.partials[(int64_t)qc * p.blocks + bc];
      x[u][k] = (q < S::kTotal && b < p.blocks) ? v : 0.0;
    }
  }
#pragma unroll
  for (int u = 0; u < kPerWave; ++u) {
    const int q = wave + 16 * u;
    double v = 0.0;
#pragma unroll
    for (int k = 0; k < kPerLane; ++k) v += x[u][k];
    v = wave_sum(v);
    if (lane == 0 && q < S::kTotal) tot[q] = v;
  }
  __syncthreads();
  // the searches run on wave 0: lane k evaluates grid point k
  if (wave != 0) return;
  ClipResult r;
  const double nan = __builtin_nan("");
  r.l_new = p.l_old;
  r.h_new = p.h_old;
  r.l_star = r.h_star = r.alpha_low = r.rho_bf16 = r.rho_fp8 = nan;
  r.n_neg = (int64_t)tot[0];
  r.n_pos = (int64_t)tot[1];
  r.l_updated = r.h_updated = 0;
  if (r.n_neg > 0) {
    const int64_t cnt_ref = (int64_t)tot[2];
    r.alpha_low = (double)cnt_ref / (double)r.n_neg;
    // #(r_FP8 <= L_k) = the negative tokens in bins 0 .. k; the first k
    // with the least distance wins (key: distance, then k)
    uint64_t key = ~0ull;
    // (the counts are exact in float64, so their prefix sums are too)
    const int64_t below = (int64_t)prefix_in_order(tot + S::kCount, p.nl);
    if (lane < p.nl) {
      const int64_t d = below > cnt_ref ? below - cnt_ref : cnt_ref - below;
      key = ((uint64_t)d << 8) | (uint64_t)lane;
    }
    key = wave_min_u64(key);
    const int kl = (int)(key & 0xff);
    r.l_star = grid_point(p.l_min, p.step, kl);
    r.l_new = smooth_update(p.l_old, r.l_star, p.delta_l);
    r.l_updated = 1;
    // Eq. 5 denominator at L*: the negative tokens with r_FP8 > L*, bins
    // kl + 1 .. nl, in bin order
    double den = 0.0;
    {
      const double v = lane <= p.nl ? tot[S::kDen + lane] : 0.0;
      for (int j = kl + 1; j <= p.nl; ++j) den += readlane_f64(v, j);
    }
    den = fabs(den);
    const double den_ref = fabs(tot[4]);
    if (den_ref > 0.0 && den > 0.0) {
      const double rho_ref = fabs(tot[3]) / den_ref;
      r.rho_bf16 = rho_ref;
      // numerator at H_k: the positive tokens with r_FP8 < H_k, bins 0 ..
      // k in order; the distance is non-negative, so its bit pattern orders
      // like its value
      double rho = 0.0;
      uint64_t dbits = ~0ull;
      const double num = prefix_in_order(tot + S::kNum, p.nh);
      if (lane < p.nh) {
        rho = fabs(num) / den;
        dbits = __double_as_longlong(fabs(rho - rho_ref));
      }
      const uint64_t dmin = wave_min_u64(dbits);
      const uint64_t first = __ballot(lane < p.nh && dbits == dmin);
      const int kh = (int)__builtin_ctzll(first);
      r.h_star = grid_point(p.h_min, p.step, kh);
      r.rho_fp8 = __shfl(rho, kh, 64);
      r.h_new = smooth_update(p.h_old, r.h_star, p.delta_h);
      r.h_updated = 1;
    } else if (den_ref > 0.0) {
      r.rho_bf16 = fabs(tot[3]) / den_ref;
    }
  }
  if (lane == 0) *p.result = r;
}

template <int KL, int KH, int T>
hipError_t launch(const ClipArgs& p, hipStream_t s) {
  clip_stats_kernel<KL, KH, T><<<p.blocks, T, 0, s>>>(p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  clip_search_kernel<KL, KH><<<1, 1024, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace clip_detail

int clip_slots(int nl, int nh) {
  if (nl <= 21 && nh <= 41) return clip_detail::Slots<21, 41>::kTotal;
  if (nl <= kClipMaxL && nh <= kClipMaxH) return clip_detail::Slots<kClipMaxL, kClipMaxH>::kTotal;
  return -1;
}

hipError_t launch_calibrate_clip(const ClipArgs& p, hipStream_t s) {
  // the paper's grids (21 and 41 points) get their own instantiation; any
  // grid up to kClipMaxL / kClipMaxH points takes the general one; 768
  // threads a block (three waves per SIMD)
  if (p.nl <= 21 && p.nh <= 41) return clip_detail::launch<21, 41, 768>(p, s);
  return clip_detail::launch<kClipMaxL, kClipMaxH, 768>(p, s);
}

// The partial sums of the allocation-free entry point: room for the most
// blocks a batch is split into and the largest grids, on every device the
// library runs on, for the life of the process.  In host code `scratch`
// only stands in for the symbol: its device address comes from
// hipGetSymbolAddress, once per device, and only that address is used.
static __device__ __align__(256) double scratch[kClipScratchBytes / sizeof(double)];
static_assert(kClipScratchBytes ==
                  (int64_t)kClipMaxBlocks * clip_detail::Slots<kClipMaxL, kClipMaxH>::kTotal * sizeof(double),
              "the scratch holds the partials of kClipMaxBlocks blocks at the largest grids");

hipError_t clip_scratch(hipStream_t s, double** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static double* addr[kMaxDevices] = {};
  int cur = 0, dev = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  dev = cur;
  if (s) {
    e = hipStreamGetDevice(s, &dev);
    if (e != hipSuccess) return e;
  }
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    // the lookup runs with the stream's device current (each device holds
    // its own copy of the array at its own address)
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = static_cast<double*>(p);
  }
  *ptr = addr[dev];
  return hipSuccess;
}

}  // namespace fp8q
