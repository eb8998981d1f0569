// Global top-B selection (Sec. 5.2 last paragraph, Algorithm 1 phase 3) and
// the retained-row plan of eq. problem, one workgroup per (sequence, head).
//
// Scores map to order-preserving uint32 keys (NaN -> -inf, -0 -> +0). An
// MSB-first radix select finds the key tau of the B-th largest prunable
// score and how many tokens equal to tau must be kept; it starts below the
// bits that every candidate shares (from the block's key min and max, or from
// a lower bound for tau and the max) and takes 11-bit digits, so scores
// spanning a few binades need up to three passes. The
// write-out walks positions in order: tokens above tau are kept, tokens equal
// to tau are kept while their rank among equals is below that count (lower
// positions first), protected tokens are always kept. Histogram increments are
// aggregated per wave with ballots (scores cluster by step utility, so most
// lanes of a wave share a digit) before the LDS atomics.
//
// Sequences of up to 32768 tokens keep their keys in registers (32 per
// thread, position tid + 1024 j in slot j); longer ones re-read the scores
// in every pass. In a batch of 2 to 64 sequences the workgroups take the
// rows of the longest sequences first. The work per key is plain VALU arithmetic over lane data;
// per-slot lane masks are made where they are used, never held across a
// phase, since 32 of them do not fit the scalar registers.
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

// In registers, a protected token holds this key: above every score's key
// (+inf maps to 0xFF800000), so it is kept by the same test as a score above
// tau; positions past the sequence hold 0. Neither is a candidate.
constexpr uint32_t kProtKey = 0xFFFFFFFFu;
// No score maps to key 1 (it would be a NaN's), so `key == 1` is never a tie.
constexpr uint32_t kNoKey = 1u;

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

// Exclusive prefix sum over the workgroup in thread order (modulo 2^32).
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* scratch) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t x = (uint32_t)__shfl_up((int)inc, o, kWave);
    if (lane >= o) inc += x;
  }
  if (lane == 63) scratch[wave] = inc;
  __syncthreads();
  uint32_t before = 0u;
  for (int w = 0; w < wave; ++w) before += scratch[w];
  __syncthreads();
  return before + inc - v;
}

// Kept candidates of one slot grouped by step: one atomic per step per wave.
__device__ __forceinline__ void count_kept_steps(int32_t* kept, int nsteps, int k, int lane) {
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

// Candidate count and key range over the workgroup in one barrier round.
// hist[0..kBins) is cleared before the same barrier for the first pass.
__device__ __forceinline__ void reduce_count_range(int& npr, uint32_t& kmin, uint32_t& kmax,
                                                   uint32_t (*red)[kWaves], uint32_t* hist) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int e = threadIdx.x; e < kBins; e += kThreads) hist[e] = 0u;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, o, kWave));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, o, kWave));
  }
  if (lane == 0) {
    red[0][wave] = (uint32_t)npr;
    red[1][wave] = kmin;
    red[2][wave] = kmax;
  }
  __syncthreads();
  npr = 0;
  for (int w = 0; w < kWaves; ++w) {
    npr += (int)red[0][w];
    kmin = min(kmin, red[1][w]);
    kmax = max(kmax, red[2][w]);
  }
}

// MSB-first radix search for the key tau of the ktake-th largest candidate
// (kmin..kmax: candidate key range, kmin < kmax) and the number `need` of
// tokens equal to tau that are kept. count(h, pmask, prefix, shift, nbins)
// adds each candidate key with (key & pmask) == prefix to bin
// (key >> shift) & (nbins - 1) of h. Two histograms alternate: each pass
// counts into one and clears the other, which only the previous pass read;
// the first must be clear and visible on entry.
template <typename Count>
__device__ __forceinline__ void radix_search(uint32_t kmin, uint32_t kmax, int ktake,
                                             uint32_t* hist, int* sh, Count count, uint32_t& tau,
                                             int& need) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int lo = 32 - __builtin_clz(kmin ^ kmax);  // undecided low bits
  const uint32_t low = lo == 32 ? 0xFFFFFFFFu : ((1u << lo) - 1u);
  uint32_t pmask = ~low;
  uint32_t prefix = kmax & pmask;
  int krem = ktake;
  int buf = 0;
  while (lo > 0) {
    const int width = min(kDigitBits, lo);
    const int shift = lo - width;
    const int nbins = 1 << width;
    uint32_t* h = hist + buf * kBins;
    uint32_t* hn = hist + (buf ^ 1) * kBins;
    for (int e = tid; e < kBins; e += kThreads) hn[e] = 0u;
    count(h, pmask, prefix, shift, nbins);
    __syncthreads();
    if (wave == 0) {
      // lane owns bins 32*lane .. 32*lane+31 (bins >= nbins stay zero);
      // find the bin holding the krem-th largest key
      constexpr int kPer = kBins / kWave;
      int b0 = kPer * lane;
      asm volatile("" : "+v"(b0));  // bin numbers made here, not held across passes
      const uint4* hp = reinterpret_cast<const uint4*>(h + b0);
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
          sh[0] = bin;
          sh[1] = krem - (int)above;
        }
        above += c;
      };
#pragma unroll
      for (int q = kPer / 4 - 1; q >= 0; --q) {  // bins from high to low
        const uint4 h4 = hp[q];
        visit(h4.w, b0 + 4 * q + 3);
        visit(h4.z, b0 + 4 * q + 2);
        visit(h4.y, b0 + 4 * q + 1);
        visit(h4.x, b0 + 4 * q);
      }
    }
    __syncthreads();
    prefix |= (uint32_t)sh[0] << shift;
    pmask |= (uint32_t)(nbins - 1) << shift;
    krem = sh[1];
    lo = shift;
    buf ^= 1;
  }
  tau = prefix;
  need = krem;  // tokens equal to tau that are kept, lowest positions first
}

struct RowSetup {
  int s, lh, seq0, ns, B, nsteps;
  int32_t* kept;
};

// Rows of the sequence of rank q when the sequences are ordered by decreasing
// length (equal lengths by index), for batches of 2 to 64 sequences:
// workgroups are dispatched in block order, so the rows of the longest
// sequences start first and the shortest fill the end of the launch. Every
// wave computes it from one round of loads of the sequence offsets.
__device__ __forceinline__ void longest_first(const SelectArgs& a, int q, RowSetup& r) {
  const int lane = threadIdx.x & 63;
  const bool in = lane < a.S;
  const int c0 = in ? a.cu_seqlens[lane] : 0;
  const int len = in ? a.cu_seqlens[lane + 1] - c0 : -1;
  int rank = 0;
  for (int j = 0; j < a.S; ++j) {
    const int lj = __shfl(len, j, kWave);
    rank += (lj > len || (lj == len && j < lane)) ? 1 : 0;
  }
  // ranks are a permutation of 0 .. S-1
  r.s = uniform(__builtin_ctzll(ballot(in && rank == q)));
  r.seq0 = uniform(__shfl(c0, r.s, kWave));
  r.ns = uniform(__shfl(len, r.s, kWave));
}

__device__ __forceinline__ RowSetup row_setup(const SelectArgs& a) {
  RowSetup r;
  const int q = blockIdx.x / a.LH;
  r.lh = blockIdx.x - q * a.LH;
  if (a.S > 1 && a.S <= kWave) {
    longest_first(a, q, r);
  } else {
    r.s = q;
    r.seq0 = a.cu_seqlens[r.s];
    r.ns = a.cu_seqlens[r.s + 1] - r.seq0;
  }
  r.B = a.budgets ? max(1, a.budgets[r.s]) : a.budget;
  const int st0 = a.kept ? a.cu_steps[r.s] : 0;
  r.nsteps = a.kept ? a.cu_steps[r.s + 1] - st0 : 0;
  r.kept = a.kept ? a.kept + (size_t)r.lh * a.total_steps + st0 : nullptr;
  if (r.kept) {
    for (int k = threadIdx.x; k < r.nsteps; k += kThreads) r.kept[k] = 0;
    __threadfence();  // the zeros reach L2 before any wave's atomics below
  }
  return r;
}

// Protected tokens of sequence s, counted by the whole workgroup: 16 at a
// time from aligned 16-byte words, the unaligned head and tail one byte at a
// time.
__device__ int count_protected(const SelectArgs& a, int s, int* scratch) {
  const int seq0 = a.cu_seqlens[s], ns = a.cu_seqlens[s + 1] - seq0;
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
  return block_sum_int(np, scratch);
}

__device__ __forceinline__ int budget_of(const SelectArgs& a, int s) {
  return a.budgets ? max(1, a.budgets[s]) : a.budget;
}

// cu_retained[s+1] - cu_retained[s] = n_protected_s + min(B_s, N_s - n_protected_s)
// Without heads there are no selection workgroups; one workgroup writes the plan.
__global__ __launch_bounds__(kThreads) void retained_plan_kernel(SelectArgs a) {
  __shared__ int scratch[kWaves];
  int acc = 0;
  if (threadIdx.x == 0) a.cu_retained[0] = 0;
  for (int s = 0; s < a.S; ++s) {
    const int ns = a.cu_seqlens[s + 1] - a.cu_seqlens[s];
    const int np = count_protected(a, s, scratch);
    acc += np + min(budget_of(a, s), ns - np);
    if (threadIdx.x == 0) a.cu_retained[s + 1] = acc;
  }
}

// The same plan from the selection workgroups of head 0: the workgroup of
// sequence s counts the protected tokens of the sequences before it (none
// with a single sequence) before it loads its keys, and adds its own
// sequence once its candidate count npr = N_s - n_protected_s is known.
// Block-uniform: only the head-0 workgroups call these.
__device__ int retained_before(const SelectArgs& a, int s, int* scratch) {
  int acc = 0;
  for (int t = 0; t < s; ++t) {
    const int nt = a.cu_seqlens[t + 1] - a.cu_seqlens[t];
    const int np = count_protected(a, t, scratch);
    acc += np + min(budget_of(a, t), nt - np);
  }
  return acc;
}

__device__ __forceinline__ void write_retained(const SelectArgs& a, int s, int before, int ns,
                                               int npr, int B) {
  if (threadIdx.x == 0) {
    if (s == 0) a.cu_retained[0] = 0;
    a.cu_retained[s + 1] = before + (ns - npr) + min(B, npr);
  }
}

// The M-th largest candidate key among a thread's slots, 0 when it holds
// fewer than M candidates (candidate keys are never 0).
template <int M>
__device__ __forceinline__ uint32_t mth_largest(const uint32_t (&keys)[kCached]) {
  uint32_t top[M];  // the largest so far, in descending order
#pragma unroll
  for (int q = 0; q < M; ++q) top[q] = 0u;
#pragma unroll
  for (int j = 0; j < kCached; ++j) {
    uint32_t x = keys[j] - 1u < kProtKey - 1u ? keys[j] : 0u;
#pragma unroll
    for (int q = 0; q < M; ++q) {
      const uint32_t hi = max(top[q], x);
      x = min(top[q], x);
      top[q] = hi;
    }
  }
  return top[M - 1];
}

// ---------------------------------------------------------------- N_s <= 32768
__global__ __launch_bounds__(kThreads) void select_cached_kernel(SelectArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t hist[2 * kBins];
  __shared__ uint32_t red[5][kWaves];
  __shared__ int sh[2];
  __shared__ int plan_scratch[kWaves];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const RowSetup r = row_setup(a);
  const int ns = r.ns;
  const float* __restrict__ P = a.scores + (size_t)r.lh * a.ntot + r.seq0;
  const uint8_t* __restrict__ prot = a.prot + r.seq0;
  const int plan_before = r.lh == 0 ? retained_before(a, r.s, plan_scratch) : 0;

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
  uint32_t keys[kCached];
  int npr = 0;  // wave total
  uint32_t kmin1 = 0xFFFFFFFFu, kmax1 = 0u;  // candidate key - 1 and + 1
#pragma unroll
  for (int j = 0; j < kCached; ++j) {
    // NaN -> -inf and -0 -> +0 in float arithmetic, then the sign flip
    const float q = fmaxf(pv[j], -INFINITY) + 0.0f;
    const uint32_t u = __float_as_uint(q);
    const uint32_t key = u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
    const bool in = tid + kThreads * j < ns;
    keys[j] = in ? (pb[j] == 0u ? key : kProtKey) : 0u;
    // key - 1 wraps 0 to the top and puts kProtKey just below it
    const uint32_t km = keys[j] - 1u;
    npr += __popcll(ballot(km < kProtKey - 1u));
    kmin1 = min(kmin1, km);
    kmax1 = max(kmax1, keys[j] + 1u);  // kProtKey + 1 wraps to 0
  }
  // A lower bound for tau: each thread holding at least m candidates has m
  // of them at or above its m-th largest, so at least m times as many
  // candidates as there are such threads lie at or above the smallest of
  // those m-th largest keys; when ktake is within that number, tau lies there
  // too and the search skips every key below it. m = 1, 2 or 4, the least
  // for which the budget can be within the bound.
  const int m = r.B <= kThreads ? 1 : (r.B <= 2 * kThreads ? 2 : 4);
  uint32_t mth;  // this thread's m-th largest candidate key, 0 with fewer than m
  if (m == 1) {
    mth = kmax1 >= 2u ? kmax1 - 1u : 0u;
  } else {
    mth = m == 2 ? mth_largest<2>(keys) : mth_largest<4>(keys);
  }
  const bool has = mth != 0u;
  uint32_t tmax = has ? mth : 0xFFFFFFFFu;
  const int nthr = __popcll(ballot(has));  // wave total
  // count, key range and the bound, reduced in one barrier round; kmin1 and
  // kmax1 in the shifted domains, where non-candidates lose every min and max
  for (int e = tid; e < kBins; e += kThreads) hist[e] = 0u;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kmin1 = min(kmin1, (uint32_t)__shfl_xor((int)kmin1, o, kWave));
    kmax1 = max(kmax1, (uint32_t)__shfl_xor((int)kmax1, o, kWave));
    tmax = min(tmax, (uint32_t)__shfl_xor((int)tmax, o, kWave));
  }
  if (lane == 0) {
    red[0][wave] = (uint32_t)npr;
    red[1][wave] = kmin1;
    red[2][wave] = kmax1;
    red[3][wave] = tmax;
    red[4][wave] = (uint32_t)nthr;
  }
  __syncthreads();
  npr = 0;
  int nthr_all = 0;
  for (int w = 0; w < kWaves; ++w) {
    npr += (int)red[0][w];
    kmin1 = min(kmin1, red[1][w]);
    kmax1 = max(kmax1, red[2][w]);
    tmax = min(tmax, red[3][w]);
    nthr_all += (int)red[4][w];
  }
  const uint32_t kmin = kmin1 + 1u, kmax = kmax1 - 1u;  // used only when there are candidates
  const int ktake = min(r.B, npr);
  const bool take_all = ktake == npr;
  if (r.lh == 0) write_retained(a, r.s, plan_before, ns, npr, r.B);

  uint32_t tau = 0u;
  int need = 0;
  if (!take_all) {
    const uint32_t lbound = ktake <= m * nthr_all ? tmax : kmin;  // tau >= lbound
    if (lbound == kmax) {
      tau = kmax;  // every candidate from the bound up ties
      need = ktake;
    } else {
      const uint32_t span = kmax - lbound;
      auto count = [&](uint32_t* h, uint32_t pmask, uint32_t prefix, int shift, int nbins) {
        // fresh compares in every pass rather than lane masks held across passes
#pragma unroll
        for (int j = 0; j < kCached; ++j) asm volatile("" : "+v"(keys[j]));
        const uint32_t dm = (uint32_t)(nbins - 1);
        // keys in [lbound, kmax] only: 0 and kProtKey fall outside
#pragma unroll
        for (int j = 0; j < kCached; ++j)
          wave_hist_add(h, keys[j] - lbound <= span && (keys[j] & pmask) == prefix,
                        (keys[j] >> shift) & dm, lane);
      };
      radix_search(lbound, kmax, ktake, hist, sh, count, tau, need);
    }
  }

  // ---- ordered write-out. Ranks in position order straight from the
  // strided slots: per (slot, wave) the numbers of sure keeps and of ties,
  // one exclusive scan over the 512 (slot, wave) pairs, which are already in
  // position order, and ballots for the ranks inside a wave. A tie is kept
  // when fewer than `need` ties precede it, so the tokens kept before
  // position p are the sure keeps before p plus min(ties before p, need).
  int32_t* __restrict__ out = a.idx + (size_t)r.lh * a.ntot + r.seq0;
  const uint32_t t_sure = take_all ? 0u : tau;    // key > t_sure: kept for sure
  const uint32_t t_tie = take_all ? kNoKey : tau;  // key == t_tie: a tie
  uint32_t* cnt = hist;  // [kCached][kWaves]: sure | ties << 16
#pragma unroll
  for (int j = 0; j < kCached; ++j) asm volatile("" : "+v"(keys[j]));
#pragma unroll
  for (int j = 0; j < kCached; ++j) {
    const uint32_t c = (uint32_t)__popcll(ballot(keys[j] > t_sure)) |
                       ((uint32_t)__popcll(ballot(keys[j] == t_tie)) << 16);
    if (lane == 0) cnt[j * kWaves + wave] = c;
  }
  __syncthreads();
  // at most 32768 tokens: both halves of the packed sums stay below 2^16
  const uint32_t ex = block_exclusive_scan(tid < kCached * kWaves ? cnt[tid] : 0u, red[0]);
  if (tid < kCached * kWaves) cnt[tid] = ex;
  __syncthreads();
  const uint32_t base_lane = lane < kCached ? cnt[lane * kWaves + wave] : 0u;
#pragma unroll
  for (int j = 0; j < kCached; ++j) asm volatile("" : "+v"(keys[j]));
  const int32_t* __restrict__ sid = a.step_ids + r.seq0;
  int tid_w = tid;
  asm volatile("" : "+v"(tid_w));  // positions and addresses made here, not carried from the top
#pragma unroll
  for (int j = 0; j < kCached; ++j) {
    const bool sure = keys[j] > t_sure, tie = keys[j] == t_tie;
    const uint64_t bs = ballot(sure), bt = ballot(tie);
    if ((bs | bt) == 0ull) continue;
    const uint32_t base = (uint32_t)__builtin_amdgcn_readlane((int)base_lane, j);
    const int s_before = (int)(base & 0xFFFFu) + lanes_below(bs);
    const int t_before = (int)(base >> 16) + lanes_below(bt);
    const bool keep = sure || (tie && t_before < need);
    const int i = tid_w + kThreads * j;
    if (keep) out[s_before + min(t_before, need)] = i;
    if (r.kept) {
      const bool cand = keys[j] - 1u < kProtKey - 1u;
      count_kept_steps(r.kept, r.nsteps, (keep && cand) ? sid[i] : -1, lane);
    }
  }
}

// ---------------------------------------------------------------- N_s > 32768
// Keys are re-read from the scores in every pass; the write-out ranks one
// slot at a time with two barrier rounds per slot.
__global__ __launch_bounds__(kThreads) void select_stream_kernel(SelectArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t hist[2 * kBins];
  __shared__ uint32_t red[3][kWaves];
  __shared__ int wcnt[2][2][kWaves];
  __shared__ int sh[2];
  __shared__ int plan_scratch[kWaves];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const RowSetup r = row_setup(a);
  const int ns = r.ns;
  const float* __restrict__ P = a.scores + (size_t)r.lh * a.ntot + r.seq0;
  const uint8_t* __restrict__ prot = a.prot + r.seq0;
  const int plan_before = r.lh == 0 ? retained_before(a, r.s, plan_scratch) : 0;
  // position of slot j of this thread: tid + kThreads * j (coalesced)
  auto key_at = [&](int j) -> uint32_t {
    const int i = tid + kThreads * j;
    if (i >= ns || prot[i] != 0) return 0u;
    return order_key(P[i]);
  };
  const int nslots = (ns + kThreads - 1) / kThreads;
  int npr = 0;
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  for (int j = 0; j < nslots; ++j) {
    const uint32_t key = key_at(j);
    npr += key != 0u ? 1 : 0;
    kmin = min(kmin, key != 0u ? key : 0xFFFFFFFFu);
    kmax = max(kmax, key);
  }
  npr = wave_sum_int(npr);
  reduce_count_range(npr, kmin, kmax, red, hist);
  const int ktake = min(r.B, npr);
  const bool take_all = ktake == npr;
  if (r.lh == 0) write_retained(a, r.s, plan_before, ns, npr, r.B);

  uint32_t tau = 0u;
  int need = 0;
  if (!take_all) {
    if (kmin == kmax) {
      tau = kmin;
      need = ktake;
    } else {
      auto count = [&](uint32_t* h, uint32_t pmask, uint32_t prefix, int shift, int nbins) {
        for (int j = 0; j < nslots; ++j) {
          const uint32_t key = key_at(j);
          wave_hist_add(h, key != 0u && (key & pmask) == prefix,
                        (key >> shift) & (uint32_t)(nbins - 1), lane);
        }
      };
      radix_search(kmin, kmax, ktake, hist, sh, count, tau, need);
    }
  }

  int32_t* __restrict__ out = a.idx + (size_t)r.lh * a.ntot + r.seq0;
  const int32_t* __restrict__ sid = a.step_ids + r.seq0;
  int tie_base = 0, out_base = 0;
  for (int j = 0; j < nslots; ++j) {
    const uint32_t key = key_at(j);
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
    if (r.kept) count_kept_steps(r.kept, r.nsteps, (keep && cand) ? sid[i] : -1, lane);
  }
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t st) {
  if (a.S * a.LH == 0) {
    hipLaunchKernelGGL(retained_plan_kernel, dim3(1), dim3(kThreads), 0, st, a);
  } else {
    if (a.max_len <= kThreads * kCached)
      hipLaunchKernelGGL(select_cached_kernel, dim3(a.S * a.LH), dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL(select_stream_kernel, dim3(a.S * a.LH), dim3(kThreads), 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace stepkv
