// Test stand-ins for the kernel launchers behind the C-ABI (the functions
// abi.hip calls in quantize.hip, gemm.hip and clip.hip), for a host-only
// build of abi.hip under the sanitizers: each records its call and the
// arguments the C-ABI passed, and launches nothing.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace fp8q {

int stub_calls = 0;
int64_t stub_nscales = 0;
GemmArgs stub_gemm;
int stub_pair = -1;

hipError_t launch_quantize(const QuantArgs& a, int, bool, int64_t nscales, hipStream_t) {
  ++stub_calls;
  stub_nscales = nscales;
  (void)a;
  return hipSuccess;
}
hipError_t launch_cast_f32(const float*, int64_t, float, bool, uint8_t*, hipStream_t) {
  ++stub_calls;
  return hipSuccess;
}
hipError_t launch_quantize_dual(const DualArgs&, hipStream_t) {
  ++stub_calls;
  return hipSuccess;
}
hipError_t launch_gemm(const GemmArgs& g, int pair, int, hipStream_t) {
  ++stub_calls;
  stub_gemm = g;
  stub_pair = pair;
  return hipSuccess;
}
hipError_t launch_gemm_grouped(const GemmGroup&, int, hipStream_t) {
  ++stub_calls;
  return hipSuccess;
}
hipError_t launch_gemm_quantized(const GemmArgs& g, int, hipStream_t) {
  ++stub_calls;
  stub_gemm = g;
  return hipSuccess;
}
hipError_t launch_gemm_splitk(const GemmArgs& g, int pair, hipStream_t) {
  ++stub_calls;
  stub_gemm = g;
  stub_pair = pair;
  return hipSuccess;
}
// the real slot counts of the two instantiations of the clipping kernels
int clip_slots(int nl, int nh) {
  if (nl <= 21 && nh <= 41) return 5 + 2 * 22 + 42;
  if (nl <= kClipMaxL && nh <= kClipMaxH) return 5 + 2 * (kClipMaxL + 1) + kClipMaxH + 1;
  return -1;
}
hipError_t launch_calibrate_clip(const ClipArgs&, hipStream_t) {
  ++stub_calls;
  return hipSuccess;
}
hipError_t clip_scratch(hipStream_t, double** ptr) {
  *ptr = reinterpret_cast<double*>(static_cast<uintptr_t>(0x20000));
  return hipSuccess;
}

}  // namespace fp8q
