// Global top-B selection (Sec. 5.2 last paragraph, Algorithm 1 phase 3) and
// the retained-row plan of eq. problem, one workgroup per (sequence, head).
//
// Scores map to order-preserving uint32 keys (NaN -> -inf, -0 -> +0). An
// MSB-first radix select finds the key tau of the B-th largest prunable
// score and how many tokens equal to tau must be kept; it starts below the
// bits that every candidate shares (from the block's key min and max) and
// takes 11-bit digits, so scores spanning a few binades need three passes. The
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
  u = (u & 0x7FFFFFFFu) > 0x7F800000u ? 0xFF800000u : u;  // NaN ranks as -inf
  u = u == 0x80000000u ? 0u : u;                           // -0 ranks as +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);       // never 0 for canonical values
}

constexpr int kDigitBits = 11;
constexpr int kBins = 1 << kDigitBits;

// Add one to h[bin] for every active lane: when every active lane of the wave
// holds the same bin (scores cluster by step), one atomic adds the count;
// otherwise each active lane adds one.
__device__ __forceinline__ void wave_hist_add(uint32_t* h, bool active, uint32_t bin, int lane) {
  const uint64_t act = ballot(active);
  if (!act) return;
  const int leader = __builtin_ctzll(act);
  const uint32_t lb = __builtin_amdgcn_readlane(bin, leader);
  const uint64_t same = ballot(active && bin == lb);
  if (same == act) {
    if (lane == leader) atomicAdd(&h[lb], (uint32_t)__popcll(act));
  } else if (active) {
    atomicAdd(&h[bin], 1u);
  }
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

// Exclusive prefix sum over the workgroup in thread order; `total` gets the sum.
__device__ __forceinline__ int block_exclusive_scan(int v, int* scratch, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int x = __shfl_up(inc, o, kWave);
    if (lane >= o) inc += x;
  }
  if (lane == 63) scratch[wave] = inc;
  __syncthreads();
  int before = 0, tot = 0;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
    const int c = scratch[w];
    before += w < wave ? c : 0;
    tot += c;
  }
  __syncthreads();
  total = tot;
  return before + inc - v;
}

// Exclusive prefix sums of four counters at once over the workgroup in
// thread order; `total` gets the four sums. scratch holds 4 * waves ints.
__device__ __forceinline__ int4 block_exclusive_scan4(int4 v, int* scratch, int4& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nw = (int)(blockDim.x >> 6);
  int4 inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int4 x = make_int4(__shfl_up(inc.x, o, kWave), __shfl_up(inc.y, o, kWave),
                             __shfl_up(inc.z, o, kWave), __shfl_up(inc.w, o, kWave));
    if (lane >= o) {
      inc.x += x.x;
      inc.y += x.y;
      inc.z += x.z;
      inc.w += x.w;
    }
  }
  if (lane == 63) {
    scratch[4 * wave] = inc.x;
    scratch[4 * wave + 1] = inc.y;
    scratch[4 * wave + 2] = inc.z;
    scratch[4 * wave + 3] = inc.w;
  }
  __syncthreads();
  int4 before = make_int4(0, 0, 0, 0), tot = make_int4(0, 0, 0, 0);
  for (int w = 0; w < nw; ++w) {
    const int4 c = make_int4(scratch[4 * w], scratch[4 * w + 1], scratch[4 * w + 2],
                             scratch[4 * w + 3]);
    if (w < wave) {
      before.x += c.x;
      before.y += c.y;
      before.z += c.z;
      before.w += c.w;
    }
    tot.x += c.x;
    tot.y += c.y;
    tot.z += c.z;
    tot.w += c.w;
  }
  __syncthreads();
  total = tot;
  return make_int4(before.x + inc.x - v.x, before.y + inc.y - v.y, before.z + inc.z - v.z,
                   before.w + inc.w - v.w);
}

// cu_retained[s+1] - cu_retained[s] = n_protected_s + min(B_s, N_s - n_protected_s)
__global__ __launch_bounds__(kThreads) void retained_plan_kernel(SelectArgs a) {
  __shared__ int scratch[kWaves];
  int acc = 0;
  if (threadIdx.x == 0) a.cu_retained[0] = 0;
  for (int s = 0; s < a.S; ++s) {
    const int seq0 = a.cu_seqlens[s], ns = a.cu_seqlens[s + 1] - seq0;
    // protected flags counted 16 at a time from aligned 16-byte words; the
    // unaligned head and tail one byte at a time
    const int misal = (int)(reinterpret_cast<uintptr_t>(a.prot + seq0) & 15);
    const int head = min(ns, (16 - misal) & 15);
    const int nvec = (ns - head) / 16;
    int np = 0;
    if ((int)threadIdx.x < head) np += a.prot[seq0 + threadIdx.x] != 0;
    const uint4* vp = reinterpret_cast<const uint4*>(a.prot + seq0 + head);
    for (int i = threadIdx.x; i < nvec; i += kThreads) {
      const uint4 w = vp[i];
      const uint32_t x[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int c = 0; c < 4; ++c) {  // one bit per nonzero byte
        uint32_t b = x[c] | (x[c] >> 4);
        b |= b >> 2;
        b |= b >> 1;
        np += __builtin_popcount(b & 0x01010101u);
      }
    }
    for (int i = head + 16 * nvec + threadIdx.x; i < ns; i += kThreads) np += a.prot[seq0 + i] != 0;
    np = block_sum_int(np, scratch);
    const int B = a.budgets ? max(1, a.budgets[s]) : a.budget;
    acc += np + min(B, ns - np);
    if (threadIdx.x == 0) a.cu_retained[s + 1] = acc;
  }
}

template <bool CACHED>
__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t hist[3 * kThreads];  // histogram, then bitmasks
  __shared__ int scratch[4 * kWaves];
  __shared__ uint32_t kred[2][kWaves];
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
  uint32_t prot_bits = 0;  // bit j: position tid + 1024 j is protected
  int npr = 0;
  if (CACHED) {
    // every load issued before any is used: indices clamped into the sequence
    float pv[kCached];
    uint32_t pb[kCached];
    if (ns > 0) {
#pragma unroll
      for (int j = 0; j < kCached; ++j) {
        const int ic = min(tid + kThreads * j, ns - 1);
        pv[j] = P[ic];
        pb[j] = prot[ic];
      }
    }
#pragma unroll
    for (int j = 0; j < kCached; ++j) {
      // branch-free: selects only, so no per-slot lane masks stay live
      const uint32_t in = (uint32_t)(tid + kThreads * j - ns) >> 31;  // 1 if inside
      const uint32_t pr = in & (pb[j] != 0u ? 1u : 0u);
      const uint32_t key = order_key(pv[j]);
      keys[j] = (in & (pr ^ 1u)) ? key : 0u;
      prot_bits |= pr << j;
      npr += keys[j] != 0u ? 1 : 0;
    }
    asm volatile("" : "+v"(prot_bits));  // rebuilt from lane masks otherwise
  } else {
    for (int j = 0; j < nslots; ++j) npr += (tid + kThreads * j < ns && prot[tid + kThreads * j] == 0);
  }
  npr = block_sum_int(npr, scratch);  // also orders the kept[] zeroing before its atomics
  const int ktake = min(B, npr);
  const bool take_all = ktake == npr;

  uint32_t tau = 0u;
  int need = 0;
  if (!take_all) {
    // range of the candidate keys: bits above the highest differing bit are shared
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
    auto range = [&](uint32_t key) {
      if (key != 0u) {
        kmin = min(kmin, key);
        kmax = max(kmax, key);
      }
    };
    if (CACHED) {
#pragma unroll
      for (int j = 0; j < kCached; ++j) range(keys[j]);
    } else {
      for (int j = 0; j < nslots; ++j) range(key_at(j));
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, o, kWave));
      kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, o, kWave));
    }
    if (lane == 0) {
      kred[0][wave] = kmin;
      kred[1][wave] = kmax;
    }
    __syncthreads();
    for (int w = 0; w < kWaves; ++w) {
      kmin = min(kmin, kred[0][w]);
      kmax = max(kmax, kred[1][w]);
    }
    if (kmin == kmax) {
      tau = kmin;  // every candidate ties
      need = ktake;
    } else {
      int lo = 32 - __builtin_clz(kmin ^ kmax);  // undecided low bits
      const uint32_t low = lo == 32 ? 0xFFFFFFFFu : ((1u << lo) - 1u);
      uint32_t pmask = ~low;
      uint32_t prefix = kmax & pmask;
      int krem = ktake;
      while (lo > 0) {
        // fresh compares in every pass: otherwise the compiler keeps 32 lane
        // masks of `key != 0` alive across the passes and spills them
        if (CACHED) {
#pragma unroll
          for (int j = 0; j < kCached; ++j) asm volatile("" : "+v"(keys[j]));
        }
        const int width = min(kDigitBits, lo);
        const int shift = lo - width;
        const int nbins = 1 << width;
        for (int e = tid; e < kBins; e += kThreads) hist[e] = 0u;
        __syncthreads();
        auto count = [&](uint32_t key) {
          const bool cand = key != 0u && (key & pmask) == prefix;
          wave_hist_add(hist, cand, (key >> shift) & (uint32_t)(nbins - 1), lane);
        };
        if (CACHED) {
#pragma unroll
          for (int j = 0; j < kCached; ++j) count(keys[j]);  // slots past N hold key 0: no candidate
        } else {
          for (int j = 0; j < nslots; ++j) count(key_at(j));
        }
        __syncthreads();
        if (wave == 0) {
          // lane owns bins 32*lane .. 32*lane+31 (bins >= nbins stay zero);
          // find the bin holding the krem-th largest key
          constexpr int kPer = kBins / kWave;
          const uint4* hp = reinterpret_cast<const uint4*>(hist + kPer * lane);
          uint32_t own = 0u;
#pragma unroll
          for (int q = 0; q < kPer / 4; ++q) {
            const uint4 h4 = hp[q];
            own += (h4.x + h4.y) + (h4.z + h4.w);
          }
          uint32_t suf = own;  // inclusive suffix over lanes >= lane
#pragma unroll
          for (int o = 1; o < 64; o <<= 1) {
            const uint32_t x = __shfl_down(suf, o, kWave);
            if (lane + o < 64) suf += x;
          }
          uint32_t above = suf - own;  // keys in bins owned by higher lanes
          auto visit = [&](uint32_t c, int bin) {
            if (above < (uint32_t)krem && (uint32_t)krem <= above + c) {
              sh_digit = bin;
              sh_krem = krem - (int)above;
            }
            above += c;
          };
#pragma unroll
          for (int q = kPer / 4 - 1; q >= 0; --q) {  // bins from high to low
            const uint4 h4 = hp[q];
            visit(h4.w, kPer * lane + 4 * q + 3);
            visit(h4.z, kPer * lane + 4 * q + 2);
            visit(h4.y, kPer * lane + 4 * q + 1);
            visit(h4.x, kPer * lane + 4 * q);
          }
        }
        __syncthreads();
        prefix |= (uint32_t)sh_digit << shift;
        pmask |= (uint32_t)(nbins - 1) << shift;
        krem = sh_krem;
        lo = shift;
      }
      tau = prefix;
      need = krem;  // tokens equal to tau that are kept, lowest positions first
    }
  }

  if (CACHED) {
#pragma unroll
    for (int j = 0; j < kCached; ++j) asm volatile("" : "+v"(keys[j]));
  }
  // ---- ordered write-out
  int32_t* __restrict__ out = a.idx + (size_t)lh * a.ntot + seq0;
  const int32_t* __restrict__ sid = a.step_ids + seq0;
  if (CACHED) {
    // Flags (1 keep for sure, 2 tie with tau, 4 protected) go through LDS
    // in batches of 8192 positions so that each thread then holds a run of
    // 8 consecutive positions per batch; ordered ranks come from two
    // four-way block scans (one lane of the scan per batch).
    constexpr int kBatch = 8192, kRun = kBatch / kThreads;  // 8
    uint8_t* fstage = reinterpret_cast<uint8_t*>(hist);      // 8 KiB of the 12 KiB
    uint64_t fl[4] = {0ull, 0ull, 0ull, 0ull};
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      if (b * kBatch < ns) {
#pragma unroll
        for (int jj = 0; jj < kRun; ++jj) {
          const int j = kRun * b + jj;
          const uint32_t key = keys[j];
          const bool pr = (prot_bits >> j) & 1u;
          const bool cand = key != 0u;
          const uint32_t f = (pr || (cand && (take_all || key > tau)) ? 1u : 0u) |
                             (cand && !take_all && key == tau ? 2u : 0u) | (pr ? 4u : 0u);
          fstage[tid + kThreads * jj] = (uint8_t)f;
        }
        __syncthreads();
        fl[b] = reinterpret_cast<const uint64_t*>(fstage)[tid];  // positions b*8192 + 8 tid + r
        __syncthreads();
      }
    }
    auto count_bits = [](uint64_t f, uint64_t m) {
      return __popcll(f & m);  // one bit per byte selected by m
    };
    const uint64_t kOne = 0x0101010101010101ull;
    int4 nt = make_int4(count_bits(fl[0], 2 * kOne), count_bits(fl[1], 2 * kOne),
                        count_bits(fl[2], 2 * kOne), count_bits(fl[3], 2 * kOne));
    int4 tt;
    const int4 tb = block_exclusive_scan4(nt, scratch, tt);
    const int tie_off[4] = {tb.x, tt.x + tb.y, tt.x + tt.y + tb.z, tt.x + tt.y + tt.z + tb.w};
    // keep mask per batch run: byte r set when position 8 tid + r is kept
    uint32_t keepm[4];
    int kc[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      uint32_t m = 0u;
      int rank = tie_off[b];
#pragma unroll
      for (int r = 0; r < kRun; ++r) {
        const uint32_t f = (uint32_t)(fl[b] >> (8 * r)) & 0xFFu;
        bool keep = (f & 1u) != 0u;
        if (f & 2u) {
          keep = rank < need;  // ties: lowest positions first
          ++rank;
        }
        m |= (keep ? 1u : 0u) << r;
      }
      keepm[b] = m;
      kc[b] = __popc(m);
    }
    int4 kt;
    const int4 kb = block_exclusive_scan4(make_int4(kc[0], kc[1], kc[2], kc[3]), scratch, kt);
    const int out_off[4] = {kb.x, kt.x + kb.y, kt.x + kt.y + kb.z, kt.x + kt.y + kt.z + kb.w};
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      int off = out_off[b];
      uint32_t m = keepm[b];
      while (m) {
        const int r = __builtin_ctz(m);
        m &= m - 1u;
        out[off++] = kBatch * b + kRun * tid + r;
      }
    }
    if (kept) {
      // run-length aggregated per thread: consecutive positions share a step
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        uint32_t m = keepm[b];
        int cur = -1, cnt = 0;
        while (m) {
          const int r = __builtin_ctz(m);
          m &= m - 1u;
          if ((fl[b] >> (8 * r)) & 4ull) continue;  // protected: no step
          const int k = sid[kBatch * b + kRun * tid + r];
          if (k != cur) {
            if (cur >= 0 && cur < nsteps && cnt) atomicAdd(&kept[cur], cnt);
            cur = k;
            cnt = 0;
          }
          ++cnt;
        }
        if (cur >= 0 && cur < nsteps && cnt) atomicAdd(&kept[cur], cnt);
      }
    }
    return;
  }

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
  for (int j = 0; j < nslots; ++j) emit(j, key_at(j));
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
