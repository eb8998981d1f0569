// Pooling, normalisation and step-utility fusion (Sec. 5.2, eq. token-priority).
// Without step statistics, and with more (sequence, head) rows than CUs or
// more than 4096 steps in a sequence, each row is spread over workgroups of
// 2048 positions (prio_chunk_*). Otherwise one workgroup per (sequence,
// head). Both compute
//   U_i  = sum_{|j-i| <= half} A_j [j prunable]     (k * T_i; zero padded)
//   Th_i = U_i / max_{prunable} U                   (the 1/k cancels)
//   P_i  = alpha * Th_i + beta * S[step_ids[i]]     (prunable; -inf if protected)
// Step statistics (count, max and fixed-point sum of Th over each step's
// prunable tokens) are segmented reductions keyed by step id: partial results
// over runs of one step go to LDS atomics in unsigned fixed point, so the
// result does not depend on the order of the atomics.
//
// Fast path (N_s <= 32768, pooling window <= 9): the sequence is staged in
// LDS in batches of 8192 positions with coalesced loads; each thread pools a
// run of 8 consecutive positions from registers and keeps its 32 pooled
// values in registers for the second sweep. Otherwise the sequence streams
// through a 1024-position LDS tile.
#include "common.h"
#include "internal.h"

#include <math.h>

#include <type_traits>

namespace stepkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kMaxHalf = 31;

struct StatOut {  // layout of stepkv_step_stat
  uint32_t count;
  float max_saliency;
  uint64_t sum_q32;
};

constexpr int kWaves = kThreads / kWave;
constexpr int kBatch = 8192;             // positions staged in LDS per batch
constexpr int kRun = kBatch / kThreads;  // consecutive positions per thread per batch
constexpr int kMaxBatches = 4;           // fast path: N_s <= 32768
constexpr int kFastHalf = 4;             // fast path: pooling window <= 9

// Per-step statistics tables in dynamic LDS (after the utility table).
struct StepTables {
  float* util;
  uint32_t* cnt;
  uint32_t* mx;
  unsigned long long* sum;
};

__device__ __forceinline__ StepTables step_tables(uint8_t* dyn, int max_steps) {
  StepTables t;
  t.util = reinterpret_cast<float*>(dyn);
  t.cnt = reinterpret_cast<uint32_t*>(dyn) + max_steps;
  t.mx = t.cnt + max_steps;
  t.sum = reinterpret_cast<unsigned long long*>(dyn + ((size_t)(3 * max_steps) * 4 + 7) / 8 * 8);
  return t;
}

__device__ __forceinline__ void flush_stat(const StepTables& t, int k, uint32_t cnt, float mx,
                                           float sum) {
  atomicAdd(&t.cnt[k], cnt);
  atomicMax(&t.mx[k], __float_as_uint(mx));  // Th >= 0: bit order = value order
  atomicAdd(&t.sum[k], (unsigned long long)((double)sum * 4294967296.0 + 0.5));
}

__device__ __forceinline__ void write_stats(const FuseArgs& a, const StepTables& t, int lh,
                                            int st0, int nsteps) {
  StatOut* so = reinterpret_cast<StatOut*>(a.stats) + (size_t)lh * a.total_steps + st0;
  for (int k = threadIdx.x; k < nsteps; k += kThreads) {
    StatOut r;
    r.count = t.cnt[k];
    r.max_saliency = __uint_as_float(t.mx[k]);
    r.sum_q32 = t.sum[k];
    so[k] = r;
  }
}

// FLAGS: the conditions of STEPKV_FLAG_* are checked and reported (only when
// the caller passed a status word; the unchecked instantiation carries none of it).
template <int HALF, bool FLAGS>
__global__ __launch_bounds__(kThreads) void fuse_batched_kernel(FuseArgs a) {
  // stage[kFastHalf + p] holds batch position p; runs of 8 positions are read
  // as aligned 16-byte vectors, global traffic stays coalesced (tid + 1024 j)
  __shared__ __attribute__((aligned(16))) float stage[kFastHalf + kBatch + kFastHalf];
  __shared__ __attribute__((aligned(16))) uint8_t pstage[kBatch];  // prunable flags
  __shared__ float wred[kWaves];
  extern __shared__ uint8_t dyn[];

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
  const bool stats = a.stats != nullptr;
  const StepTables tabs = step_tables(dyn, a.max_steps);
  for (int k = tid; k < nsteps; k += kThreads) {
    tabs.util[k] = a.util[st0 + k];
    if (stats) {
      tabs.cnt[k] = 0u;
      tabs.mx[k] = 0u;
      tabs.sum[k] = 0ull;
    }
  }
  const int nb = (ns + kBatch - 1) / kBatch;
  constexpr int J = kRun * kMaxBatches;  // 32 coalesced slots: position tid + 1024 j

  // every A and protected-flag load of the sequence, issued up front
  float x[J];
  uint32_t pb[J];
  if (ns > 0) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int ic = min(tid + kThreads * j, ns - 1);
      x[j] = A[ic];
      pb[j] = prot[ic];
    }
  }
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const bool pr = ns > 0 && tid + kThreads * j < ns && pb[j] == 0;
    x[j] = pr ? x[j] : 0.f;
    pb[j] = pr ? 1u : 0u;
  }

  float u[kMaxBatches][kRun];
  uint32_t prun = 0u;  // bit kRun*b + r: position b*kBatch + kRun*tid + r is prunable
  float mloc = 0.f;    // U >= 0, and Th = 0 everywhere when the max is 0
#pragma unroll
  for (int b = 0; b < kMaxBatches; ++b) {
    if (b < nb) {
#pragma unroll
      for (int jj = 0; jj < kRun; ++jj) {
        stage[kFastHalf + tid + kThreads * jj] = x[kRun * b + jj];
        pstage[tid + kThreads * jj] = (uint8_t)pb[kRun * b + jj];
      }
      // halos: the 4 positions before the batch sit in the previous batch's last
      // slot of threads 1020..1023, the 4 after it in the next batch's first slot
      if (tid >= kThreads - kFastHalf)
        stage[tid - (kThreads - kFastHalf)] = b > 0 ? x[b > 0 ? kRun * b - 1 : 0] : 0.f;
      if (tid < kFastHalf)
        stage[kFastHalf + kBatch + tid] = b + 1 < kMaxBatches ? x[b + 1 < kMaxBatches ? kRun * (b + 1) : 0] : 0.f;
      __syncthreads();
      // run: positions kRun*tid - 4 .. kRun*tid + 11 of the batch
      float v[16];
      const float4* sp = reinterpret_cast<const float4*>(stage + kRun * tid);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 f = sp[q];
        v[4 * q] = f.x;
        v[4 * q + 1] = f.y;
        v[4 * q + 2] = f.z;
        v[4 * q + 3] = f.w;
      }
      const uint64_t fl = *reinterpret_cast<const uint64_t*>(&pstage[kRun * tid]);
#pragma unroll
      for (int r = 0; r < kRun; ++r) {
        float acc = 0.f;
#pragma unroll
        for (int o = 0; o <= 2 * HALF; ++o) acc += v[kFastHalf - HALF + r + o];
        u[b][r] = acc;
        const bool pr = (fl >> (8 * r)) & 0xFFull;
        prun |= (pr ? 1u : 0u) << (kRun * b + r);
        mloc = pr ? fmaxf(mloc, acc) : mloc;
      }
      __syncthreads();  // the next batch reuses the stage
    }
  }
  mloc = wave_max(mloc);
  if (lane == 0) wred[wave] = mloc;
  // step ids of the sequence, coalesced, issued while the maximum is reduced
  int32_t sv[J];
  if (ns > 0) {
#pragma unroll
    for (int j = 0; j < J; ++j) sv[j] = sid[min(tid + kThreads * j, ns - 1)];
  }
  __syncthreads();
  float M = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wred[w]);
  const float inv = M > 0.f ? 1.0f / M : 0.f;

  // ---- sweep 2: normalise, fuse; the run's scores go back through the stage
  float* __restrict__ out = a.scores + (size_t)lh * a.ntot + seq0;
  int32_t* istage = reinterpret_cast<int32_t*>(stage);
  // wave masks of the conditions met (STEPKV_FLAG_*): a prunable token with an
  // out-of-range step id, or a non-finite priority (non-finite saliency or utility)
  uint64_t bad_id = 0ull, bad_nf = 0ull;
#pragma unroll
  for (int b = 0; b < kMaxBatches; ++b) {
    if (b < nb) {
#pragma unroll
      for (int jj = 0; jj < kRun; ++jj) istage[tid + kThreads * jj] = sv[kRun * b + jj];
      __syncthreads();
      const int4 k0 = reinterpret_cast<const int4*>(istage + kRun * tid)[0];
      const int4 k1 = reinterpret_cast<const int4*>(istage + kRun * tid)[1];
      const int kr[kRun] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
      float pv[kRun];
      int cur = -1;
      uint32_t ccount = 0u;
      float cmax = 0.f, csum = 0.f;
#pragma unroll
      for (int r = 0; r < kRun; ++r) {
        const bool pr = (prun >> (kRun * b + r)) & 1u;
        const int kk = kr[r];
        const bool ok = pr && kk >= 0 && kk < nsteps;
        const float th = u[b][r] * inv;
        const float util = ok ? tabs.util[ok ? kk : 0] : 0.f;
        pv[r] = pr ? fmaf(a.alpha, th, a.beta * util) : -INFINITY;
        if (FLAGS) {
          bad_id |= __ballot(pr && !ok);
          bad_nf |= __ballot(pr && !finite(pv[r]));
        }
        if (stats) {
          const int key = ok ? kk : -1;
          if (key != cur) {
            if (cur >= 0) flush_stat(tabs, cur, ccount, cmax, csum);
            cur = key;
            ccount = 0u;
            cmax = 0.f;
            csum = 0.f;
          }
          if (key >= 0) {
            ++ccount;
            cmax = fmaxf(cmax, th);
            csum += th;
          }
        }
      }
      if (stats && cur >= 0) flush_stat(tabs, cur, ccount, cmax, csum);
      __syncthreads();  // step ids read before the stage takes the scores
      float4* wp = reinterpret_cast<float4*>(stage + kRun * tid);
      wp[0] = make_float4(pv[0], pv[1], pv[2], pv[3]);
      wp[1] = make_float4(pv[4], pv[5], pv[6], pv[7]);
      __syncthreads();
#pragma unroll
      for (int jj = 0; jj < kRun; ++jj) {
        const int i = b * kBatch + tid + kThreads * jj;
        if (i < ns) out[i] = stage[tid + kThreads * jj];
      }
      __syncthreads();  // the next batch reuses the stage
    }
  }
  if (FLAGS) report_masks(a.status, bad_id, bad_nf);
  if (stats) {
    __syncthreads();
    write_stats(a, tabs, lh, st0, nsteps);
  }
}

// General path: the sequence streams through a 1024-position tile.
__global__ __launch_bounds__(kThreads) void fuse_stream_kernel(FuseArgs a) {
  __shared__ float tile[kThreads + 2 * kMaxHalf];
  __shared__ float wred[kWaves];
  extern __shared__ uint8_t dyn[];

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
  const StepTables tabs = step_tables(dyn, a.max_steps);
  for (int k = tid; k < nsteps; k += kThreads) {
    tabs.util[k] = a.util[st0 + k];
    if (stats) {
      tabs.cnt[k] = 0u;
      tabs.mx[k] = 0u;
      tabs.sum[k] = 0ull;
    }
  }
  auto masked = [&](int j) -> float {
    return (j >= 0 && j < ns && prot[j] == 0) ? A[j] : 0.f;
  };
  auto pooled = [&](int base) -> float {
    tile[tid + half] = masked(base + tid);
    if (tid < half) tile[tid] = masked(base - half + tid);
    if (tid < half) tile[kThreads + half + tid] = masked(base + kThreads + tid);
    __syncthreads();
    float acc = 0.f;
    for (int o = 0; o <= 2 * half; ++o) acc += tile[tid + o];
    __syncthreads();
    return acc;
  };
  float mloc = 0.f;
  for (int base = 0; base < ns; base += kThreads) {
    const float uu = pooled(base);
    const int i = base + tid;
    if (i < ns && prot[i] == 0) mloc = fmaxf(mloc, uu);
  }
  mloc = wave_max(mloc);
  if (lane == 0) wred[wave] = mloc;
  __syncthreads();
  float M = 0.f;
  for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wred[w]);
  const float inv = M > 0.f ? 1.0f / M : 0.f;
  float* __restrict__ out = a.scores + (size_t)lh * a.ntot + seq0;
  uint32_t bad = 0u;  // STEPKV_FLAG_* conditions met by this thread
  for (int base = 0; base < ns; base += kThreads) {
    const float uu = pooled(base);
    const int i = base + tid;
    int kk = -1;
    float th = 0.f;
    if (i < ns) {
      const bool pr = prot[i] == 0;
      kk = sid[i];
      const bool ok = pr && kk >= 0 && kk < nsteps;
      th = uu * inv;
      const float util = ok ? tabs.util[kk] : 0.f;
      // a non-finite prunable saliency makes every pooled value around it non-finite
      bad |= (pr && !ok ? kFlagStepId : 0u) |
             (pr && !(finite(uu) && finite(util)) ? kFlagNonFinite : 0u);
      out[i] = pr ? fmaf(a.alpha, th, a.beta * util) : -INFINITY;
      if (!ok) kk = -1;
    }
    if (stats) {
      // one wave ballot per distinct step id present in the wave
      uint64_t pending = ballot(kk >= 0);
      while (pending) {
        const int leader = __builtin_ctzll(pending);
        const int key = __builtin_amdgcn_readlane(kk, leader);
        const uint64_t grp = ballot(kk == key);
        const float mine = (kk == key) ? th : 0.f;
        const float sum = wave_sum(mine);
        const float mx = wave_max(mine);
        if (lane == leader) flush_stat(tabs, key, (uint32_t)__popcll(grp), mx, sum);
        pending &= ~grp;
      }
    }
  }
  report_flags(a.status, bad);
  if (stats) {
    __syncthreads();
    write_stats(a, tabs, lh, st0, nsteps);
  }
}

}  // namespace

namespace {

// Shared-index mode: A_i = sum of the window saliency of `heads` (layer, KV
// head) rows, added in row order (deterministic). Coalesced: consecutive
// threads read consecutive tokens of each row; eight rows' loads are in
// flight before their adds.
__global__ __launch_bounds__(256) void sum_heads_kernel(const float* __restrict__ sal, int heads,
                                                        int ntot, float* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= ntot) return;
  float acc = sal[i];
  int h = 1;
  for (; h + 8 <= heads; h += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = sal[(size_t)(h + u) * ntot + i];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
  }
  for (; h < heads; ++h) acc += sal[(size_t)h * ntot + i];
  out[i] = acc;
}

// Shared-index mode without step statistics: the single priority row of each
// sequence is spread over workgroups of kShChunk positions instead of one
// workgroup per sequence. shared_sum_pool_kernel sums the heads (as
// sum_heads_kernel does), pools its chunk and writes the chunk's maximum of
// the pooled prunable values; shared_fuse_kernel takes each sequence's
// maximum from its chunks' maxima, pools again from the summed saliency and
// writes P. Both pool in the same order as fuse_batched_kernel (left to
// right from 0), so the maximum and the values agree bit for bit with it.
constexpr int kShChunk = 256;

// Chunk g of the concatenated per-sequence chunk lists: sequence s, chunk c.
__device__ __forceinline__ void shared_chunk(const int32_t* __restrict__ cu_seqlens, int S, int g,
                                             int& s, int& c, int& cfirst) {
  int acc = 0;
  s = S;
  c = 0;
  cfirst = 0;
  for (int t = 0; t < S; ++t) {
    const int n = cu_seqlens[t + 1] - cu_seqlens[t];
    const int k = (n + kShChunk - 1) / kShChunk;
    if (g < acc + k) {
      s = t;
      c = g - acc;
      cfirst = acc;
      return;
    }
    acc += k;
  }
}

// Masked (prunable) summed saliency of the chunk and its halos into am[0 ..
// kShChunk + 2 half): am[e] is position p0 - half + e of the sequence.
template <bool FROM_HEADS>
__device__ __forceinline__ void shared_stage(const SharedPrioArgs& a, int seq0, int ns, int p0,
                                             float* am, float* sum_out) {
  const int half = a.half;
  for (int e = threadIdx.x; e < kShChunk + 2 * half; e += kShChunk) {
    const int p = p0 - half + e;
    float v = 0.f;
    if (p >= 0 && p < ns) {
      const int i = seq0 + p;
      float acc;
      if (FROM_HEADS) {  // rows added in row order, eight loads in flight
        acc = a.heads[i];
        int h = 1;
        for (; h + 8 <= a.nheads; h += 8) {
          float w[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) w[u] = a.heads[(size_t)(h + u) * a.ntot + i];
#pragma unroll
          for (int u = 0; u < 8; ++u) acc += w[u];
        }
        for (; h < a.nheads; ++h) acc += a.heads[(size_t)h * a.ntot + i];
        if (e >= half && e < half + kShChunk) sum_out[i] = acc;
      } else {
        acc = a.sal[i];
      }
      v = a.prot[i] == 0 ? acc : 0.f;
    }
    am[e] = v;
  }
}

__global__ __launch_bounds__(kShChunk) void shared_sum_pool_kernel(SharedPrioArgs a) {
  __shared__ float am[kShChunk + 2 * kMaxHalf];
  __shared__ float wred[kShChunk / kWave];
  int s, c, cfirst;
  shared_chunk(a.cu_seqlens, a.S, blockIdx.x, s, c, cfirst);
  if (s >= a.S) return;  // uniform: the grid holds exactly the chunks
  const int seq0 = a.cu_seqlens[s], ns = a.cu_seqlens[s + 1] - seq0;
  const int p0 = c * kShChunk;
  shared_stage<true>(a, seq0, ns, p0, am, a.sal);
  __syncthreads();
  const int p = p0 + (int)threadIdx.x;
  float u = 0.f;
  for (int o = 0; o <= 2 * a.half; ++o) u += am[threadIdx.x + o];
  const bool pr = p < ns && a.prot[seq0 + p] == 0;
  const float m = wave_max(pr ? u : 0.f);  // U >= 0
  if ((threadIdx.x & 63) == 0) wred[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    float mm = 0.f;
    for (int w = 0; w < kShChunk / kWave; ++w) mm = fmaxf(mm, wred[w]);
    a.cmax[blockIdx.x] = mm;
  }
}

__global__ __launch_bounds__(kShChunk) void shared_fuse_kernel(SharedPrioArgs a) {
  __shared__ float am[kShChunk + 2 * kMaxHalf];
  __shared__ float wred[kShChunk / kWave];
  int s, c, cfirst;
  shared_chunk(a.cu_seqlens, a.S, blockIdx.x, s, c, cfirst);
  if (s >= a.S) return;
  const int seq0 = a.cu_seqlens[s], ns = a.cu_seqlens[s + 1] - seq0;
  const int nch = (ns + kShChunk - 1) / kShChunk;
  const int p0 = c * kShChunk;
  // the sequence's maximum over its chunks' maxima
  float m = 0.f;
  for (int k = threadIdx.x; k < nch; k += kShChunk) m = fmaxf(m, a.cmax[cfirst + k]);
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) wred[threadIdx.x >> 6] = m;
  shared_stage<false>(a, seq0, ns, p0, am, nullptr);
  __syncthreads();
  float M = 0.f;
  for (int w = 0; w < kShChunk / kWave; ++w) M = fmaxf(M, wred[w]);
  const float inv = M > 0.f ? 1.0f / M : 0.f;
  const int p = p0 + (int)threadIdx.x;
  uint32_t bad = 0u;
  if (p < ns) {
    float u = 0.f;
    for (int o = 0; o <= 2 * a.half; ++o) u += am[threadIdx.x + o];
    const int i = seq0 + p;
    const bool pr = a.prot[i] == 0;
    const int st0 = a.cu_steps[s], nsteps = a.cu_steps[s + 1] - st0;
    const int kk = a.step_ids[i];
    const bool ok = pr && kk >= 0 && kk < nsteps;
    const float util = ok ? a.util[st0 + kk] : 0.f;
    bad = (pr && !ok ? kFlagStepId : 0u) | (pr && !(finite(u) && finite(util)) ? kFlagNonFinite : 0u);
    a.scores[i] = pr ? fmaf(a.alpha, u * inv, a.beta * util) : -INFINITY;
  }
  report_flags(a.status, bad);
}

// Per-head priority without step statistics: each (layer, KV head) row is
// spread over workgroups of kPrChunk positions instead of one workgroup per
// (sequence, row), in three launches. The chunk maxima live in the scores
// row itself, at each chunk's first position, until the last launch
// overwrites them:
//   prio_chunk_max_kernel  pools its chunk, writes the chunk's maximum of the
//                          pooled prunable values at the chunk's first position
//   prio_row_max_kernel    per (sequence, row): the maximum over its chunks,
//                          written back to every chunk's first position
//   prio_chunk_fuse_kernel reads that maximum from its own chunk's first
//                          position (before anyone writes there), pools again
//                          and writes P
// Pooling adds the window left to right from its first position, as
// fuse_batched_kernel does, so U, its maximum and P agree with it bit for bit.
constexpr int kPrThreads = 256;
constexpr int kPrChunk = 2048;  // positions per workgroup, 8 per thread

// Sequence s and chunk c of global chunk g (chunks of the sequences in
// order): a wave-wide prefix over 64 sequences at a time, in every wave.
__device__ __forceinline__ void locate_chunk(const int32_t* __restrict__ cu_seqlens, int S, int g,
                                             int& s_out, int& c_out) {
  const int lane = threadIdx.x & 63;
  int base = 0;
  for (int s0 = 0; s0 < S; s0 += kWave) {
    const int sq = s0 + lane;
    const int cnt = sq < S ? (cu_seqlens[sq + 1] - cu_seqlens[sq] + kPrChunk - 1) / kPrChunk : 0;
    int incl = cnt;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int o = __shfl_up(incl, off, kWave);
      if (lane >= off) incl += o;
    }
    const int total = __shfl(incl, kWave - 1, kWave);
    if (g < base + total) {
      const int first = __builtin_ctzll(ballot(base + incl > g));
      s_out = s0 + first;
      c_out = g - base - __shfl(incl - cnt, first, kWave);
      return;
    }
    base += total;
  }
  s_out = -1;  // not reached for g below the chunk count
  c_out = 0;
}

// (layer, KV head) rows per workgroup of the spread path: the rows share the
// chunk's lookup, protected flags and step ids, and both rows' loads are in
// flight at once (4 rows, with half the workgroups resident, measured slower).
constexpr int kPrRows = 2;

// The chunk's stage in LDS: am[i][e] = A of row lh0 + i at position
// p0 - half + e of the sequence when that position exists and is prunable,
// else 0, and pf[e] = 1 for such a prunable position; e < kPrChunk + 2 half.
// Rows past LH stage zeros. Every load is issued before the first LDS write.
// A chunk whose halos lie inside the sequence (all but the first and last of
// a sequence) takes a path without clamps or range tests: the kernels are
// bound by vector instructions, most of them address arithmetic.
struct PrioStage {
  float am[kPrRows][kPrChunk + 2 * kMaxHalf];
  uint8_t pf[kPrChunk + 2 * kMaxHalf];
};

__device__ __forceinline__ void prio_stage(const FuseArgs& a, const float* const (&rowp)[kPrRows],
                                           const uint8_t* __restrict__ prot, int ns, int p0,
                                           PrioStage& st) {
  constexpr int J = kPrChunk / kPrThreads;
  const int tid = threadIdx.x;
  const int q0 = p0 - a.half;  // position of stage entry 0
  const int n_st = kPrChunk + 2 * a.half;
  float v[kPrRows][J + 1];
  uint32_t pr[J + 1];
  if (q0 >= 0 && q0 + n_st <= ns) {  // interior chunk (uniform)
#pragma unroll
    for (int j = 0; j <= J; ++j) {
      const int e = tid + kPrThreads * j;
      const int q = q0 + min(e, n_st - 1);  // slot J: only the halo past the chunk is staged
      pr[j] = prot[q];
#pragma unroll
      for (int i = 0; i < kPrRows; ++i) v[i][j] = rowp[i][q];
    }
#pragma unroll
    for (int j = 0; j <= J; ++j) {
      const int e = tid + kPrThreads * j;
      if (j < J || e < n_st) {
        const bool in = pr[j] == 0;
        st.pf[e] = in;
#pragma unroll
        for (int i = 0; i < kPrRows; ++i) st.am[i][e] = in ? v[i][j] : 0.f;
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j <= J; ++j) {
      const int e = tid + kPrThreads * j;
      const int q = min(max(q0 + e, 0), max(ns - 1, 0));
      pr[j] = prot[q];
#pragma unroll
      for (int i = 0; i < kPrRows; ++i) v[i][j] = rowp[i][q];
    }
#pragma unroll
    for (int j = 0; j <= J; ++j) {
      const int e = tid + kPrThreads * j;
      if (j < J || e < n_st) {
        const int q = q0 + e;
        const bool in = q >= 0 && q < ns && pr[j] == 0;
        st.pf[e] = in;
#pragma unroll
        for (int i = 0; i < kPrRows; ++i) st.am[i][e] = in ? v[i][j] : 0.f;
      }
    }
  }
}

// U at position p0 + e (e < kPrChunk) from the stage: the 2 half + 1 values
// around it, added left to right.
template <int HALF>
__device__ __forceinline__ float prio_pool(const float* am, int e, int half) {
  float acc = 0.f;
  if constexpr (HALF >= 0) {
#pragma unroll
    for (int o = 0; o <= 2 * HALF; ++o) acc += am[e + o];
  } else {
    for (int o = 0; o <= 2 * half; ++o) acc += am[e + o];
  }
  return acc;
}

// The workgroup's rows and chunk: row group blockIdx / total_chunks (rows
// lh0 .. lh0 + kPrRows - 1, pointers clamped to a real row past LH, whose
// values the kernels never store), chunk g of the concatenated sequences.
struct PrioWork {
  int lh0, s, seq0, ns, p0;
};

__device__ __forceinline__ bool prio_work(const FuseArgs& a, PrioWork& w) {
  const int rgrp = blockIdx.x / a.total_chunks, g = blockIdx.x - rgrp * a.total_chunks;
  int s, c;
  locate_chunk(a.cu_seqlens, a.S, g, s, c);
  s = uniform(s);
  if (s < 0) return false;
  w.lh0 = rgrp * kPrRows;
  w.s = s;
  w.seq0 = uniform(a.cu_seqlens[s]);
  w.ns = uniform(a.cu_seqlens[s + 1]) - w.seq0;
  w.p0 = uniform(c) * kPrChunk;
  return true;
}

template <int HALF>
__global__ __launch_bounds__(kPrThreads) void prio_chunk_max_kernel(FuseArgs a) {
  __shared__ PrioStage st;
  __shared__ float wred[kPrRows][kPrThreads / kWave];
  PrioWork w;
  if (!prio_work(a, w)) return;
  const float* rowp[kPrRows];
#pragma unroll
  for (int i = 0; i < kPrRows; ++i)
    rowp[i] = a.sal + (size_t)min(w.lh0 + i, a.LH - 1) * a.ntot + w.seq0;
  prio_stage(a, rowp, a.prot + w.seq0, w.ns, w.p0, st);
  __syncthreads();
  constexpr int J = kPrChunk / kPrThreads;
#pragma unroll
  for (int i = 0; i < kPrRows; ++i) {
    float m = 0.f;  // U >= 0; positions past the sequence are not prunable in pf
#pragma unroll
    for (int r = 0; r < J; ++r) {
      const int e = threadIdx.x + kPrThreads * r;
      if (st.pf[e + a.half]) m = fmaxf(m, prio_pool<HALF>(st.am[i], e, a.half));
    }
    m = wave_max(m);
    if ((threadIdx.x & 63) == 0) wred[i][threadIdx.x >> 6] = m;
  }
  __syncthreads();
  if (threadIdx.x < kPrRows && w.lh0 + (int)threadIdx.x < a.LH) {
    const int i = threadIdx.x;
    float mm = 0.f;
    for (int k = 0; k < kPrThreads / kWave; ++k) mm = fmaxf(mm, wred[i][k]);
    a.scores[(size_t)(w.lh0 + i) * a.ntot + w.seq0 + w.p0] = mm;
  }
}

__global__ __launch_bounds__(kWave) void prio_row_max_kernel(FuseArgs a) {
  const int lh = blockIdx.x / a.S, s = blockIdx.x - lh * a.S;
  const int seq0 = a.cu_seqlens[s], ns = a.cu_seqlens[s + 1] - seq0;
  const int nch = (ns + kPrChunk - 1) / kPrChunk;
  float* row = a.scores + (size_t)lh * a.ntot + seq0;
  float m = 0.f;
  for (int c = threadIdx.x; c < nch; c += kWave) m = fmaxf(m, row[(size_t)c * kPrChunk]);
  m = wave_max(m);
  for (int c = threadIdx.x; c < nch; c += kWave) row[(size_t)c * kPrChunk] = m;
}

template <int HALF, bool FLAGS>
__global__ __launch_bounds__(kPrThreads) void prio_chunk_fuse_kernel(FuseArgs a) {
  static_assert(kPrRows == 2, "the fuse loop is written for two rows");
  __shared__ PrioStage st;
  PrioWork w;
  if (!prio_work(a, w)) return;
  const float* rowp[kPrRows];
  float* outp[kPrRows];
  float M[kPrRows];  // each row's maximum; read before the barrier below
#pragma unroll
  for (int i = 0; i < kPrRows; ++i) {
    const size_t row = (size_t)min(w.lh0 + i, a.LH - 1) * a.ntot + w.seq0;
    rowp[i] = a.sal + row;
    outp[i] = a.scores + row;
    M[i] = outp[i][w.p0];
  }
  const int st0 = uniform(a.cu_steps[w.s]), nsteps = uniform(a.cu_steps[w.s + 1]) - st0;
  const int32_t* sid = a.step_ids + w.seq0;
  const float* util = a.util + st0;
  constexpr int J = kPrChunk / kPrThreads;
  const int nout = min(kPrChunk, w.ns - w.p0);  // positions of this chunk
  int32_t kv[J];  // step ids of this thread's positions
#pragma unroll
  for (int r = 0; r < J; ++r) kv[r] = sid[w.p0 + min((int)threadIdx.x + kPrThreads * r, nout - 1)];
  prio_stage(a, rowp, a.prot + w.seq0, w.ns, w.p0, st);
  __syncthreads();  // every thread has the maxima before position p0 takes its P
  float inv[kPrRows];
#pragma unroll
  for (int i = 0; i < kPrRows; ++i) inv[i] = M[i] > 0.f ? 1.0f / M[i] : 0.f;
  const bool two = w.lh0 + 1 < a.LH;  // uniform: the group's second row exists
  uint32_t bad = 0u;
#pragma unroll
  for (int r = 0; r < J; ++r) {
    const int e = threadIdx.x + kPrThreads * r;
    if (e < nout) {
      const bool pr = st.pf[e + a.half] != 0;
      const int kk = kv[r];
      const bool ok = pr && (uint32_t)kk < (uint32_t)nsteps;
      const float bu = a.beta * (ok ? util[kk] : 0.f);  // as the per-sequence kernels
      const int p = w.p0 + e;
      const float pv0 = pr ? fmaf(a.alpha, prio_pool<HALF>(st.am[0], e, a.half) * inv[0], bu)
                           : -INFINITY;
      outp[0][p] = pv0;
      float pv1 = 0.f;
      if (two) {
        pv1 = pr ? fmaf(a.alpha, prio_pool<HALF>(st.am[1], e, a.half) * inv[1], bu) : -INFINITY;
        outp[1][p] = pv1;
      }
      if (FLAGS)
        bad |= (pr && !ok ? kFlagStepId : 0u) |
               (pr && !(finite(pv0) && finite(pv1)) ? kFlagNonFinite : 0u);
    }
  }
  if (FLAGS) report_flags(a.status, bad);
}

}  // namespace

int shared_chunks(const int32_t* cu_seqlens_host, int S) {
  int n = 0;
  for (int t = 0; t < S; ++t) n += (cu_seqlens_host[t + 1] - cu_seqlens_host[t] + kShChunk - 1) / kShChunk;
  return n;
}

hipError_t launch_shared_priority(const SharedPrioArgs& a, int chunks, hipStream_t st) {
  if (chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(shared_sum_pool_kernel, dim3(chunks), dim3(kShChunk), 0, st, a);
  hipLaunchKernelGGL(shared_fuse_kernel, dim3(chunks), dim3(kShChunk), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_sum_heads(const float* sal, int heads, int ntot, float* out, hipStream_t st) {
  if (ntot == 0 || heads == 0) return hipSuccess;
  hipLaunchKernelGGL(sum_heads_kernel, dim3((ntot + 255) / 256), dim3(256), 0, st, sal, heads,
                     ntot, out);
  return hipGetLastError();
}

int prio_chunks(const int32_t* cu_seqlens_host, int S) {
  int n = 0;
  for (int t = 0; t < S; ++t) n += (cu_seqlens_host[t + 1] - cu_seqlens_host[t] + kPrChunk - 1) / kPrChunk;
  return n;
}

hipError_t launch_fuse(const FuseArgs& a, hipStream_t st) {
  if (a.S * a.LH == 0) return hipSuccess;
  // Without statistics, and when the (sequence, row) pairs outnumber the CUs
  // (the per-sequence kernel runs one 1024-thread workgroup per CU, so it
  // would take several rounds), each row is spread over workgroups of
  // kPrChunk positions. Measured on MI355X: 28 layers x 4 heads x 16 ragged
  // sequences 152 -> 118 us; with one round (32 x 8 rows of one 32k sequence)
  // the per-sequence kernel stays ahead, 37 against 41 us.
  // Sequences with more than 4096 steps take the spread path too: the
  // per-sequence kernels stage every step utility in LDS.
  if (!a.stats && (a.S * a.LH > 256 || a.max_steps > 4096)) {
    if (a.total_chunks == 0) return hipSuccess;
    const unsigned row_groups = (unsigned)((a.LH + kPrRows - 1) / kPrRows);
    const dim3 grid(row_groups * (unsigned)a.total_chunks);
    auto go = [&](auto half_c) {
      constexpr int H = decltype(half_c)::value;
      hipLaunchKernelGGL(prio_chunk_max_kernel<H>, grid, dim3(kPrThreads), 0, st, a);
      hipLaunchKernelGGL(prio_row_max_kernel, dim3((unsigned)a.LH * (unsigned)a.S), dim3(kWave), 0,
                         st, a);
      if (a.status)
        hipLaunchKernelGGL((prio_chunk_fuse_kernel<H, true>), grid, dim3(kPrThreads), 0, st, a);
      else
        hipLaunchKernelGGL((prio_chunk_fuse_kernel<H, false>), grid, dim3(kPrThreads), 0, st, a);
    };
    switch (a.half) {  // the usual pooling windows (1 .. 9) unrolled
      case 0: go(std::integral_constant<int, 0>{}); break;
      case 1: go(std::integral_constant<int, 1>{}); break;
      case 2: go(std::integral_constant<int, 2>{}); break;
      case 3: go(std::integral_constant<int, 3>{}); break;
      case 4: go(std::integral_constant<int, 4>{}); break;
      default: go(std::integral_constant<int, -1>{}); break;
    }
    return hipGetLastError();
  }
  size_t dyn = (size_t)a.max_steps * 4;
  if (a.stats) dyn = ((size_t)(3 * a.max_steps) * 4 + 7) / 8 * 8 + (size_t)a.max_steps * 8;
  const dim3 grid(a.S * a.LH), block(kThreads);
  if (a.max_len <= kBatch * kMaxBatches && a.half <= kFastHalf) {
    auto go = [&](auto half_c, auto flags_c) {
      hipLaunchKernelGGL((fuse_batched_kernel<decltype(half_c)::value, decltype(flags_c)::value>),
                         grid, block, dyn, st, a);
    };
    auto with_half = [&](auto flags_c) {
      switch (a.half) {
        case 0: go(std::integral_constant<int, 0>{}, flags_c); break;
        case 1: go(std::integral_constant<int, 1>{}, flags_c); break;
        case 2: go(std::integral_constant<int, 2>{}, flags_c); break;
        case 3: go(std::integral_constant<int, 3>{}, flags_c); break;
        default: go(std::integral_constant<int, 4>{}, flags_c); break;
      }
    };
    if (a.status) with_half(std::true_type{});
    else with_half(std::false_type{});
  } else {
    hipLaunchKernelGGL(fuse_stream_kernel, grid, block, dyn, st, a);
  }
  return hipGetLastError();
}

}  // namespace stepkv
