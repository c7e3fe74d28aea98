// probe.hip - device characterisation: the bf16 MFMA rate this GPU sustains.
//
// Not part of the method.  Every wave issues `iters` rounds of four
// independent v_mfma_f32_32x32x16_bf16 (four accumulators, so consecutive
// MFMAs never wait on each other) and nothing else in its loop; timing a
// launch that fills the chip gives the dense bf16 MFMA throughput at the
// clock the card actually runs at under MFMA load, a ceiling to hold the
// attention kernel against beside the published peak.
#include "internal.h"

namespace ditango {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(kProbeThreads) void mfma_probe_kernel(float* sink, int iters) {
  const int tid = threadIdx.x;
  // operands derived from the lane id so nothing folds at compile time;
  // small values keep the accumulators finite for any iteration count
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)((float)((tid + e) & 7) * (1.0f / 1024.0f));
    b[e] = (__bf16)((float)((tid * 3 + e) & 7) * (1.0f / 1024.0f));
  }
  f32x16 c0{}, c1{}, c2{}, c3{};
  for (int i = 0; i < iters; ++i) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
  sink[(int64_t)blockIdx.x * kProbeThreads + tid] = s;
}

}  // namespace

hipError_t launch_probe_mfma(int n_workgroups, int iters, float* sink, hipStream_t s) {
  hipLaunchKernelGGL(mfma_probe_kernel, dim3((unsigned)n_workgroups), dim3(kProbeThreads), 0, s, sink,
                     iters);
  return hipGetLastError();
}

}  // namespace ditango
