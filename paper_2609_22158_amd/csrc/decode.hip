// One decode step over the compacted cache, used to check that C_hat is a
// usable KV cache: out = softmax(scale * q . K_hat^T) V_hat for every
// (layer, sequence, query head), fp32 accumulation. A correctness check, not
// a tuned attention kernel.
#include "common.h"
#include "internal.h"

#include <math.h>

namespace stepkv {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float bf16_to_float(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

template <int D>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeArgs a) {
  constexpr int kParts = kThreads / D;
  __shared__ float q[D];
  __shared__ float e[kThreads];
  __shared__ float part[kThreads];
  __shared__ float scratch[kThreads / kWave];
  const int tid = threadIdx.x;
  const int hq = blockIdx.x % a.Hq;
  const int s = (blockIdx.x / a.Hq) % a.S;
  const int l = blockIdx.x / (a.Hq * a.S);
  const int lh = l * a.Hkv + hq / a.G;
  const int r0 = a.cu_retained[s];
  const int r1 = min(a.cu_retained[s + 1], a.out_rows);
  const int R = max(0, r1 - r0);
  const uint16_t* kb = a.k + ((size_t)lh * a.out_rows + r0) * D;
  const uint16_t* vb = a.v + ((size_t)lh * a.out_rows + r0) * D;
  const uint16_t* qp = a.q + (((size_t)l * a.S + s) * a.Hq + hq) * D;
  for (int d = tid; d < D; d += kThreads) q[d] = bf16_to_float(qp[d]);
  __syncthreads();

  auto logit = [&](int r) {
    float acc = 0.f;
    for (int d = 0; d < D; ++d) acc = fmaf(q[d], bf16_to_float(kb[(size_t)r * D + d]), acc);
    return acc * a.scale;
  };
  // max and sum of exp over the R rows
  float m = -INFINITY;
  for (int r = tid; r < R; r += kThreads) m = fmaxf(m, logit(r));
  m = wave_max(m);
  if ((tid & 63) == 0) scratch[tid >> 6] = m;
  __syncthreads();
  float M = -INFINITY;
  for (int w = 0; w < kThreads / kWave; ++w) M = fmaxf(M, scratch[w]);
  __syncthreads();
  float z = 0.f;
  for (int r = tid; r < R; r += kThreads) z += expf(logit(r) - M);
  z = wave_sum(z);
  if ((tid & 63) == 0) scratch[tid >> 6] = z;
  __syncthreads();
  float Z = 0.f;
  for (int w = 0; w < kThreads / kWave; ++w) Z += scratch[w];

  // weighted value sum, 256 rows per batch
  const int dim = tid % D, p = tid / D;
  float acc = 0.f;
  for (int b0 = 0; b0 < R; b0 += kThreads) {
    __syncthreads();
    const int r = b0 + tid;
    e[tid] = r < R ? expf(logit(r) - M) : 0.f;
    __syncthreads();
    const int nb = min(kThreads, R - b0);
    for (int rr = p; rr < nb; rr += kParts)
      acc = fmaf(e[rr], bf16_to_float(vb[(size_t)(b0 + rr) * D + dim]), acc);
  }
  part[tid] = acc;
  __syncthreads();
  if (tid < D) {
    float t = 0.f;
    for (int q2 = 0; q2 < kParts; ++q2) t += part[q2 * D + tid];
    a.out[(((size_t)l * a.S + s) * a.Hq + hq) * D + tid] = R > 0 ? t / Z : 0.f;
  }
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)(a.L * a.S * a.Hq));
  if (a.d == 128)
    hipLaunchKernelGGL(decode_kernel<128>, grid, dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(decode_kernel<64>, grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace stepkv
