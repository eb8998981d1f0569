// Issue-rate probe (a measurement, not part of the method): how much of the
// matrix cores' issue rate the saliency sweeps' instruction mix leaves. Per
// v_mfma_f32_32x32x16_bf16 (a 32 x 32 score tile over 16 of the d entries)
// the sweeps do the per-element vector work of two score elements: the scaled
// logit (v_fma_f32), its exp2 (v_exp_f32, a transcendental) and the running
// sum (v_add_f32). mix = 0 issues the MFMAs alone, mix = 1 the MFMAs with that
// work between them, each wave over four independent accumulators (and eight
// independent vector chains), so neither stream waits on its own results.
#include "common.h"
#include "internal.h"

namespace stepkv {
namespace {

constexpr int kProbeThreads = 256;

template <int MIX>
__global__ __launch_bounds__(kProbeThreads) void issue_probe_kernel(int iters, float* sink) {
  float x[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = 1e-3f * (float)(i + 1) + 1e-6f * (float)threadIdx.x;
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.5f + 0.125f * (float)i);
    b[i] = (__bf16)(0.25f - 0.0625f * (float)i);
  }
  f32x16_t acc[4] = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[m], 0, 0, 0);
      if constexpr (MIX == 1) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          float& v = x[2 * m + e];
          asm volatile("v_fma_f32 %0, %0, %0, %0" : "+v"(v));
          asm volatile("v_exp_f32 %0, %0" : "+v"(v));
          asm volatile("v_add_f32 %0, %0, %0" : "+v"(v));
        }
      }
    }
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s += x[i];
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int j = 0; j < 16; ++j) s += acc[m][j];
  sink[(size_t)blockIdx.x * kProbeThreads + threadIdx.x] = s;
}

}  // namespace

hipError_t launch_issue_probe(int mix, int blocks, int iters, float* sink, hipStream_t st) {
  if (mix == 0)
    hipLaunchKernelGGL(issue_probe_kernel<0>, dim3(blocks), dim3(kProbeThreads), 0, st, iters,
                       sink);
  else
    hipLaunchKernelGGL(issue_probe_kernel<1>, dim3(blocks), dim3(kProbeThreads), 0, st, iters,
                       sink);
  return hipGetLastError();
}

}  // namespace stepkv
