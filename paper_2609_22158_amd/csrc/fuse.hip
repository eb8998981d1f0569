// Pooling, normalisation and step-utility fusion (Sec. 5.2, eq. token-priority)
// with segmented per-step statistics, one workgroup per (sequence, head):
//   U_i  = sum_{|j-i| <= half} A_j [j prunable]     (k * T_i; zero padded)
//   Th_i = U_i / max_{prunable} U                   (the 1/k cancels)
//   P_i  = alpha * Th_i + beta * S[step_ids[i]]     (prunable; -inf if protected)
// Step statistics (count, max and fixed-point sum of Th over each step's
// prunable tokens) use one wave ballot per distinct step id in the wave and
// LDS atomics, so the result does not depend on the order of the atomics.
#include "common.h"
#include "internal.h"

#include <math.h>

namespace stepkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kMaxHalf = 31;

struct StatOut {  // layout of stepkv_step_stat
  uint32_t count;
  float max_saliency;
  uint64_t sum_q32;
};

__global__ __launch_bounds__(kThreads) void fuse_kernel(FuseArgs a) {
  __shared__ float tile[kThreads + 2 * kMaxHalf];
  __shared__ float wred[kThreads / kWave];
  extern __shared__ uint8_t dyn[];  // per-step tables: count, max bits, q32 sum

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int s = blockIdx.x / a.LH, lh = blockIdx.x - s * a.LH;
  const int seq0 = a.cu_seqlens[s];
  const int ns = a.cu_seqlens[s + 1] - seq0;
  const int st0 = a.cu_steps[s];
  const int nsteps = a.cu_steps[s + 1] - st0;
  const float* __restrict__ A = a.sal + (size_t)lh * a.ntot + seq0;
  const uint8_t* __restrict__ prot = a.prot + seq0;
  const int32_t* __restrict__ sid = a.step_ids + seq0;
  const int half = a.half;
  const bool stats = a.stats != nullptr;

  // dynamic LDS: count[max_steps], max bits[max_steps], then 8-aligned q32 sums
  uint32_t* s_cnt = reinterpret_cast<uint32_t*>(dyn);
  uint32_t* s_max = s_cnt + a.max_steps;
  unsigned long long* s_sum =
      reinterpret_cast<unsigned long long*>(dyn + ((size_t)(2 * a.max_steps) * 4 + 7) / 8 * 8);
  if (stats) {
    for (int k = tid; k < nsteps; k += kThreads) {
      s_cnt[k] = 0u;
      s_max[k] = 0u;
      s_sum[k] = 0ull;
    }
  }

  // masked saliency A_j [j prunable], zero outside the sequence
  auto masked = [&](int j) -> float {
    return (j >= 0 && j < ns && prot[j] == 0) ? A[j] : 0.f;
  };
  // U for position base + tid, reading the tile staged for [base - half, base + 1024 + half)
  auto pooled_tile = [&](int base) -> float {
    tile[tid + half] = masked(base + tid);
    if (tid < half) tile[tid] = masked(base - half + tid);
    if (tid < half) tile[kThreads + half + tid] = masked(base + kThreads + tid);
    __syncthreads();
    float u = 0.f;
    for (int o = 0; o <= 2 * half; ++o) u += tile[tid + o];
    __syncthreads();
    return u;
  };

  // ---- sweep 1: max of U over prunable tokens
  float mloc = 0.f;  // U >= 0, and Th = 0 everywhere when the max is 0
  for (int base = 0; base < ns; base += kThreads) {
    const float u = pooled_tile(base);
    const int i = base + tid;
    if (i < ns && prot[i] == 0) mloc = fmaxf(mloc, u);
  }
  mloc = wave_max(mloc);
  if (lane == 0) wred[wave] = mloc;
  __syncthreads();
  float M = 0.f;
#pragma unroll
  for (int w = 0; w < kThreads / kWave; ++w) M = fmaxf(M, wred[w]);

  // ---- sweep 2: normalise, fuse, write, segmented statistics
  float* __restrict__ out = a.scores + (size_t)lh * a.ntot + seq0;
  for (int base = 0; base < ns; base += kThreads) {
    const float u = pooled_tile(base);
    const int i = base + tid;
    int k = -1;
    float th = 0.f;
    if (i < ns) {
      if (prot[i] == 0) {
        th = M > 0.f ? u / M : 0.f;
        k = sid[i];
        const bool ok = k >= 0 && k < nsteps;
        const float util = ok ? a.util[st0 + k] : 0.f;
        out[i] = a.alpha * th + a.beta * util;
        if (!ok) k = -1;
      } else {
        out[i] = -INFINITY;
      }
    }
    if (stats) {
      // one round per distinct step id present in this wave
      uint64_t pending = ballot(k >= 0);
      while (pending) {
        const int leader = __builtin_ctzll(pending);
        const int key = __shfl(k, leader, kWave);
        const uint64_t grp = ballot(k == key);
        const float mine = (k == key) ? th : 0.f;
        const float sum = wave_sum(mine);
        const float mx = wave_max(mine);
        if (lane == leader) {
          atomicAdd(&s_cnt[key], (uint32_t)__popcll(grp));
          atomicMax(&s_max[key], __float_as_uint(mx));  // th >= 0: bit order = value order
          atomicAdd(&s_sum[key], (unsigned long long)((double)sum * 4294967296.0 + 0.5));
        }
        pending &= ~grp;
      }
    }
  }

  if (stats) {
    __syncthreads();
    StatOut* so = reinterpret_cast<StatOut*>(a.stats) + (size_t)lh * a.total_steps + st0;
    for (int k = tid; k < nsteps; k += kThreads) {
      StatOut r;
      r.count = s_cnt[k];
      r.max_saliency = __uint_as_float(s_max[k]);
      r.sum_q32 = s_sum[k];
      so[k] = r;
    }
  }
}

}  // namespace

hipError_t launch_fuse(const FuseArgs& a, hipStream_t st) {
  if (a.S * a.LH == 0) return hipSuccess;
  size_t dyn = 0;
  if (a.stats) dyn = ((size_t)(2 * a.max_steps) * 4 + 7) / 8 * 8 + (size_t)a.max_steps * 8;
  hipLaunchKernelGGL(fuse_kernel, dim3(a.S * a.LH), dim3(kThreads), dyn, st, a);
  return hipGetLastError();
}

}  // namespace stepkv
