// Global top-B selection (Sec. 5.2 last paragraph, Algorithm 1 phase 3) and
// the retained-row plan of eq. problem, one workgroup per (sequence, head).
//
// Scores map to order-preserving uint32 keys (NaN -> -inf, -0 -> +0). An
// MSB-first radix select (four 8-bit digits) finds the key tau of the B-th
// largest prunable score and how many tokens equal to tau must be kept. The
// write-out walks positions in order: tokens above tau are kept, tokens equal
// to tau are kept while their rank among equals is below that count (lower
// positions first), protected tokens are always kept. Histogram increments are
// aggregated per wave with ballots (scores cluster by step utility, so most
// lanes of a wave share a digit) before the LDS atomics.
#include "common.h"
#include "internal.h"

namespace stepkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kCached = 32;  // keys held in registers when N_s <= 32768

__device__ __forceinline__ uint32_t order_key(float p) {
  uint32_t u = __float_as_uint(p);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) u = 0xFF800000u;  // NaN ranks as -inf
  if (u == 0x80000000u) u = 0u;                            // -0 ranks as +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);       // never 0 for canonical values
}

// Add `count` lanes' worth of `bin` increments: at most four ballot rounds
// for clustered digits, then one atomic per remaining lane.
__device__ __forceinline__ void aggregated_add(uint32_t* h, bool active, uint32_t bin, int lane) {
  uint64_t pend = ballot(active);
#pragma unroll
  for (int round = 0; round < 4; ++round) {
    if (!pend) return;
    const int leader = __builtin_ctzll(pend);
    const uint32_t lb = __shfl(bin, leader, kWave);
    const uint64_t grp = ballot(active && bin == lb);
    if (lane == leader) atomicAdd(&h[lb], (uint32_t)__popcll(grp));
    pend &= ~grp;
  }
  if ((pend >> lane) & 1ull) atomicAdd(&h[bin], 1u);
}

__device__ __forceinline__ int block_sum_int(int v, int* scratch) {
  v = wave_sum_int(v);
  if ((threadIdx.x & 63) == 0) scratch[threadIdx.x >> 6] = v;
  __syncthreads();
  int t = 0;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) t += scratch[w];
  __syncthreads();
  return t;
}

// cu_retained[s+1] - cu_retained[s] = n_protected_s + min(B_s, N_s - n_protected_s)
__global__ __launch_bounds__(kThreads) void retained_plan_kernel(SelectArgs a) {
  __shared__ int scratch[kWaves];
  int acc = 0;
  if (threadIdx.x == 0) a.cu_retained[0] = 0;
  for (int s = 0; s < a.S; ++s) {
    const int seq0 = a.cu_seqlens[s], ns = a.cu_seqlens[s + 1] - seq0;
    int np = 0;
    for (int i = threadIdx.x; i < ns; i += kThreads) np += a.prot[seq0 + i] != 0;
    np = block_sum_int(np, scratch);
    const int B = a.budgets ? max(1, a.budgets[s]) : a.budget;
    acc += np + min(B, ns - np);
    if (threadIdx.x == 0) a.cu_retained[s + 1] = acc;
  }
}

template <bool CACHED>
__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a) {
  __shared__ uint32_t hist[kWaves][256];
  __shared__ int scratch[kWaves];
  __shared__ int wcnt[2][2][kWaves];
  __shared__ int sh_digit, sh_krem;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int s = blockIdx.x / a.LH, lh = blockIdx.x - s * a.LH;
  const int seq0 = a.cu_seqlens[s];
  const int ns = a.cu_seqlens[s + 1] - seq0;
  const float* __restrict__ P = a.scores + (size_t)lh * a.ntot + seq0;
  const uint8_t* __restrict__ prot = a.prot + seq0;
  const int B = a.budgets ? max(1, a.budgets[s]) : a.budget;
  const int st0 = a.kept ? a.cu_steps[s] : 0;
  const int nsteps = a.kept ? a.cu_steps[s + 1] - st0 : 0;
  int32_t* kept = a.kept ? a.kept + (size_t)lh * a.total_steps + st0 : nullptr;
  if (kept) {
    for (int k = tid; k < nsteps; k += kThreads) kept[k] = 0;
    __threadfence();  // the zeros reach L2 before any wave's atomics below
  }

  // position of slot j of this thread: tid + kThreads * j (coalesced)
  auto key_at = [&](int j) -> uint32_t {
    const int i = tid + kThreads * j;
    if (i >= ns || prot[i] != 0) return 0u;
    return order_key(P[i]);
  };
  const int nslots = (ns + kThreads - 1) / kThreads;
  uint32_t keys[CACHED ? kCached : 1];
  int npr = 0;
  if (CACHED) {
#pragma unroll
    for (int j = 0; j < kCached; ++j) {
      keys[j] = key_at(j);
      npr += keys[j] != 0u;
    }
  } else {
    for (int j = 0; j < nslots; ++j) npr += (tid + kThreads * j < ns && prot[tid + kThreads * j] == 0);
  }
  npr = block_sum_int(npr, scratch);  // also orders the kept[] zeroing before its atomics
  const int ktake = min(B, npr);
  const bool take_all = ktake == npr;

  uint32_t tau = 0u;
  int need = 0;
  if (!take_all) {
    uint32_t prefix = 0u, pmask = 0u;
    int krem = ktake;
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int e = tid; e < kWaves * 256; e += kThreads) (&hist[0][0])[e] = 0u;
      __syncthreads();
      auto count = [&](uint32_t key) {
        const bool cand = key != 0u && (key & pmask) == prefix;
        aggregated_add(hist[wave], cand, (key >> shift) & 255u, lane);
      };
      if (CACHED) {
#pragma unroll
        for (int j = 0; j < kCached; ++j)
          if (kThreads * j < ns) count(keys[j]);
      } else {
        for (int j = 0; j < nslots; ++j) count(key_at(j));
      }
      __syncthreads();
      if (wave == 0) {
        // lane owns bins 4*lane .. 4*lane+3; find the digit holding the krem-th largest
        uint32_t c4[4];
        uint32_t own = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint32_t t = 0;
          for (int w = 0; w < kWaves; ++w) t += hist[w][4 * lane + q];
          c4[q] = t;
          own += t;
        }
        uint32_t suf = own;  // inclusive suffix over lanes >= lane
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t x = __shfl_down(suf, o, kWave);
          if (lane + o < 64) suf += x;
        }
        uint32_t above = suf - own;  // keys in bins owned by higher lanes
#pragma unroll
        for (int q = 3; q >= 0; --q) {
          if (above < (uint32_t)krem && (uint32_t)krem <= above + c4[q]) {
            sh_digit = 4 * lane + q;
            sh_krem = krem - (int)above;
          }
          above += c4[q];
        }
      }
      __syncthreads();
      prefix |= (uint32_t)sh_digit << shift;
      pmask |= 255u << shift;
      krem = sh_krem;
    }
    tau = prefix;
    need = krem;  // tokens equal to tau that are kept, lowest positions first
  }

  // ---- ordered write-out
  int32_t* __restrict__ out = a.idx + (size_t)lh * a.ntot + seq0;
  const int32_t* __restrict__ sid = a.step_ids + seq0;
  int tie_base = 0, out_base = 0;
  auto emit = [&](int j, uint32_t key) {
    const int par = j & 1;
    const int i = tid + kThreads * j;
    const bool valid = i < ns;
    const bool cand = key != 0u;
    const bool definite = (valid && prot[i] != 0) || (cand && (take_all || key > tau));
    const bool tie = cand && !take_all && key == tau;
    const uint64_t bt = ballot(tie);
    if (lane == 0) wcnt[par][0][wave] = __popcll(bt);
    __syncthreads();
    int before = 0, total = 0;
    for (int w = 0; w < kWaves; ++w) {
      const int c = wcnt[par][0][w];
      before += w < wave ? c : 0;
      total += c;
    }
    const bool keep = definite || (tie && tie_base + before + lanes_below(bt) < need);
    tie_base += total;
    const uint64_t bk = ballot(keep);
    if (lane == 0) wcnt[par][1][wave] = __popcll(bk);
    __syncthreads();
    int kb = 0, kt = 0;
    for (int w = 0; w < kWaves; ++w) {
      const int c = wcnt[par][1][w];
      kb += w < wave ? c : 0;
      kt += c;
    }
    if (keep) out[out_base + kb + lanes_below(bk)] = i;
    out_base += kt;
    if (kept) {
      const int k = (keep && cand) ? sid[i] : -1;
      const bool ok = k >= 0 && k < nsteps;
      uint64_t pend = ballot(ok);
      while (pend) {
        const int leader = __builtin_ctzll(pend);
        const int kk = __shfl(k, leader, kWave);
        const uint64_t grp = ballot(ok && k == kk);
        if (lane == leader) atomicAdd(&kept[kk], (int)__popcll(grp));
        pend &= ~grp;
      }
    }
  };
  if (CACHED) {
#pragma unroll
    for (int j = 0; j < kCached; ++j)
      if (kThreads * j < ns) emit(j, keys[j]);
  } else {
    for (int j = 0; j < nslots; ++j) emit(j, key_at(j));
  }
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(retained_plan_kernel, dim3(1), dim3(kThreads), 0, st, a);
  if (a.S * a.LH > 0) {
    if (a.max_len <= kThreads * kCached)
      hipLaunchKernelGGL(select_kernel<true>, dim3(a.S * a.LH), dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL(select_kernel<false>, dim3(a.S * a.LH), dim3(kThreads), 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace stepkv
