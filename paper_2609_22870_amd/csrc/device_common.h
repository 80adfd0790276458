// Device helpers shared by the fp8q kernels (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fp8q {

constexpr float kE4M3Max = 448.0f;     // largest finite OCP E4M3 magnitude
constexpr float kE5M2Max = 57344.0f;   // largest finite OCP E5M2 magnitude

// F_max of the code format: E4M3, or E5M2 (E5 = true, the gradient variant).
template <bool E5>
constexpr float fp8_max() { return E5 ? kE5M2Max : kE4M3Max; }

// bf16 halves of a packed dword, widened exactly to fp32.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Per-unit constants of Eq. 3: the scale S = RN32(amax / F_max) (1 if that
// is 0), its correctly rounded reciprocal, and whether the reciprocal-based
// quotient below is exact for this S.
struct UnitScale {
  float s;
  float r;
  bool fast;
};

__device__ __forceinline__ UnitScale unit_scale(float amax, float fmax = kE4M3Max) {
  UnitScale u;
  float s = amax / fmax;      // IEEE division (correctly rounded)
  u.s = (s == 0.0f) ? 1.0f : s;
  u.r = 1.0f / u.s;           // IEEE division (correctly rounded)
  u.fast = u.s >= 0x1p-90f;
  return u;
}

// The power-of-two variant: S = the smallest power of two with F_max S >=
// amax, at least 2^-127 (the E8M0 range of the matrix instructions' block
// scales), and 1 when amax is 0.  Then |x| / S <= F_max and x / S is exact.
// Both maxima are 7/8 of a power of two, 448 = (7/8) 2^9 and 57344 =
// (7/8) 2^16: with amax = m 2^e (m in [0.5, 1)), amax / F_max =
// (8 m / 7) 2^(e - p), and 8 m / 7 <= 1 exactly when m <= 7/8.
__device__ __forceinline__ UnitScale unit_scale_pow2(float amax, int p = 9) {
  UnitScale u;
  if (amax == 0.0f) {
    u.s = 1.0f;
  } else {
    int e;
    const float m = frexpf(amax, &e);
    int k = e - p + (m > 0.875f ? 1 : 0);
    k = k < -127 ? -127 : k;
    u.s = ldexpf(1.0f, k);
  }
  u.r = 1.0f / u.s;  // exact: a power of two
  u.fast = u.s >= 0x1p-90f;
  return u;
}

__device__ __forceinline__ UnitScale unit_scale(float amax, bool pow2) {
  return pow2 ? unit_scale_pow2(amax) : unit_scale(amax);
}

// The same for the code format E4M3 or E5M2.
template <bool E5>
__device__ __forceinline__ UnitScale unit_scale_fmt(float amax, bool pow2) {
  return pow2 ? unit_scale_pow2(amax, E5 ? 16 : 9) : unit_scale(amax, fp8_max<E5>());
}

// RN32(x / S) for a bf16 x of the unit whose scale is u.  For S >= 2^-90 the
// quotient is formed from the reciprocal with one residual correction,
//   q0 = RN(x r),  e = RN(q0 S - x) (one FMA),  q = RN(q0 - e r) (one FMA);
// over every pair of a bf16 amax and a bf16 x with |x| <= amax, both signs,
// this gives the same E4M3 code as the correctly rounded quotient (checked
// exhaustively on the CPU, and on the GPU against the oracle).  The residual
// is taken as q0 S - x, not x - q0 S, so that x = -0 keeps its sign: the
// exact zero residual is +0 and -(+0) r + (-0) = -0.  Smaller S take the
// IEEE division.
__device__ __forceinline__ float fast_quotient(float x, float s, float r) {
  const float q0 = x * r;
  const float e = __builtin_fmaf(q0, s, -x);
  return __builtin_fmaf(-e, r, q0);
}

__device__ __forceinline__ float quotient(float x, const UnitScale& u) {
  if (u.fast) return fast_quotient(x, u.s, u.r);
  return x / u.s;
}

// Q_FP8 of two fp32 values into the low (HI=false) or high 16 bits of
// `old`: clamp to +-448, then the hardware E4M3 conversion, which rounds to
// nearest even and keeps the sign of zero.
template <bool HI>
__device__ __forceinline__ uint32_t e4m3_pack2(float a, float b, uint32_t old) {
  float ca = __builtin_amdgcn_fmed3f(a, -kE4M3Max, kE4M3Max);
  float cb = __builtin_amdgcn_fmed3f(b, -kE4M3Max, kE4M3Max);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(ca, cb, (int)old, HI);
}

// The E5M2 form: clamp to +-57344, then the hardware E5M2 conversion (round
// to nearest even, sign of zero kept); never an infinity.
template <bool HI>
__device__ __forceinline__ uint32_t e5m2_pack2(float a, float b, uint32_t old) {
  float ca = __builtin_amdgcn_fmed3f(a, -kE5M2Max, kE5M2Max);
  float cb = __builtin_amdgcn_fmed3f(b, -kE5M2Max, kE5M2Max);
  return (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(ca, cb, (int)old, HI);
}

template <bool E5, bool HI>
__device__ __forceinline__ uint32_t fp8_pack2(float a, float b, uint32_t old) {
  return E5 ? e5m2_pack2<HI>(a, b, old) : e4m3_pack2<HI>(a, b, old);
}

// Max over the 16 lanes of a DPP row (lanes 16k .. 16k+15).  Each step
// combines a lane with a partner in the same row; after quad swaps the four
// lanes of a quad agree, the half-row mirror joins the two quads of each half,
// the row mirror joins the two halves.
__device__ __forceinline__ float row16_max(float v) {
  int b = __float_as_int(v);
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(b, b, 0xB1, 0xF, 0xF, false)));  // quad [1,0,3,2]
  b = __float_as_int(v);
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(b, b, 0x4E, 0xF, 0xF, false)));  // quad [2,3,0,1]
  b = __float_as_int(v);
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(b, b, 0x141, 0xF, 0xF, false)));  // row_half_mirror
  b = __float_as_int(v);
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(b, b, 0x140, 0xF, 0xF, false)));  // row_mirror
  return v;
}

// Max over the four DPP rows of the wave for lanes with equal (lane % 16).
__device__ __forceinline__ float across_rows_max(float v) {
  v = fmaxf(v, __shfl_xor(v, 16, 64));
  v = fmaxf(v, __shfl_xor(v, 32, 64));
  return v;
}

__device__ __forceinline__ float wave_max(float v) { return across_rows_max(row16_max(v)); }

}  // namespace fp8q
