// Device-side helpers shared by the StepKV kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace stepkv {

constexpr int kWave = 64;

typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16_t __attribute__((__vector_size__(16 * sizeof(float))));

// Wave-uniform value from lane 0 (an SGPR).
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

// Number of set bits of `mask` below this lane.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  const uint32_t lo = static_cast<uint32_t>(mask), hi = static_cast<uint32_t>(mask >> 32);
  return __builtin_amdgcn_mbcnt_hi(hi, __builtin_amdgcn_mbcnt_lo(lo, 0u));
}

// ORs the STEPKV_FLAG_* bits that any lane of the wave met into the device
// status word (one atomic per wave, none when no lane met a condition). Every
// lane of the wave must reach the call.
__device__ __forceinline__ void report_flags(uint32_t* status, uint32_t bits) {
  if (status == nullptr) return;
  uint32_t w = 0u;
#pragma unroll
  for (uint32_t b = 1u; b <= 4u; b <<= 1) w |= __ballot((bits & b) != 0u) ? b : 0u;
  if (w != 0u && (threadIdx.x & (kWave - 1)) == __builtin_ctzll(__ballot(1)))
    atomicOr(status, w);
}

// x is neither NaN nor infinite.
__device__ __forceinline__ bool finite(float x) { return fabsf(x) <= 3.40282347e38f; }

// ORs the STEPKV_FLAG_* bits of wave-wide condition masks (ballots kept in
// scalar registers while the wave works) into the device status word: one
// atomic per wave, none when no lane met a condition. Wave-uniform call.
__device__ __forceinline__ void report_masks(uint32_t* status, uint64_t step_id_mask,
                                             uint64_t nonfinite_mask) {
  const uint32_t w = (step_id_mask ? 1u : 0u) | (nonfinite_mask ? 2u : 0u);
  if (status != nullptr && w != 0u &&
      (threadIdx.x & (kWave - 1)) == __builtin_ctzll(__ballot(1)))
    atomicOr(status, w);
}

// Wait until at most N vector memory operations of this wave are outstanding
// (they complete in issue order; direct-to-LDS loads count too).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `ahead` tiles of NLD loads each are still in flight
// (ahead = tiles issued after the one needed next, 0 <= ahead <= MAXA).
template <int NLD, int MAXA>
__device__ __forceinline__ void wait_tiles(int ahead) {
  if constexpr (MAXA <= 0) {
    wait_vmem<0>();
  } else {
    if (ahead >= MAXA) wait_vmem<MAXA * NLD>();
    else wait_tiles<NLD, MAXA - 1>(ahead);
  }
}

// Pins x to this point of the program: the compiler must have x here (it
// waits for the load that produced it here, once, instead of at a first use
// inside a tile loop, where the wait would also drain a prefetch ring), and
// cannot sink the computation of x past this point.
template <typename T>
__device__ __forceinline__ void settle(T& x) {
  asm volatile("" : "+v"(x));
}

// 2^x on the transcendental unit (v_exp_f32); -inf gives 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Index of the last entry of the non-decreasing array cu[0..n] that is <= x,
// for cu[0] <= x < cu[n] (the segment holding x).
__device__ __forceinline__ int segment_of(const int32_t* __restrict__ cu, int n, int x) {
  int lo = 0, hi = n;  // invariant: cu[lo] <= x < cu[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cu[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

}  // namespace stepkv
