// One decode step over the compacted cache C_hat: out = softmax(scale *
// q . K_hat^T) V_hat for every (layer, sequence, query head), fp32
// accumulation (the consumer of the compacted cache, Sec. 3).
//
// decode_mfma_kernel: one workgroup per (layer, KV head, sequence, split of
// 512 retained rows) serves all G <= 16 query heads of the KV head, so K and V
// are read once: q . k for the whole query group on MFMA, an exact online
// softmax per head, p V in fp32 on the vector units; decode_combine_kernel
// merges the splits. decode_simple_kernel serves groups wider than 16 heads.
#include "common.h"
#include "internal.h"

#include <math.h>

#include <algorithm>
#include <type_traits>

namespace stepkv {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float bf16_to_float(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Retained rows [r0, r0 + R) of sequence s, clamped to [0, out_rows) so that
// no cu_retained value leads a read out of the cache.
__device__ __forceinline__ int rows_of(const DecodeArgs& a, int s, int& r0) {
  r0 = min(max(a.cu_retained[s], 0), a.out_rows);
  return min(max(a.cu_retained[s + 1], r0), a.out_rows) - r0;
}

template <int D>
__global__ __launch_bounds__(kThreads) void decode_simple_kernel(DecodeArgs a) {
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
  if (blockIdx.x == 0 && tid == 0 && a.status && a.cu_retained[a.S] > a.out_rows)
    atomicOr(a.status, kFlagOutRows);  // rows past out_rows are not read
  int r0;
  const int R = rows_of(a, s, r0);
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


#ifndef STEPKV_DECODE_SPLIT_ROWS
#define STEPKV_DECODE_SPLIT_ROWS 512
#endif
constexpr int kSplitRows = STEPKV_DECODE_SPLIT_ROWS;  // retained rows per workgroup

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void unpack8(const u32x4_t& w, float (&f)[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

// Row splits of sequence s: ceil(R_s / kSplitRows).
__device__ __forceinline__ int splits_of(const DecodeArgs& a, int s) {
  int r0;
  return (rows_of(a, s, r0) + kSplitRows - 1) / kSplitRows;
}

// The sequence holding global split gs, and the first global split of that
// sequence: a wave-wide prefix sum over 64 sequences at a time. s_out = -1
// when gs is past the last split (the grid is sized by a host-side bound).
__device__ __forceinline__ void locate_split(const DecodeArgs& a, int gs, int& s_out,
                                             int& first_out) {
  const int lane = threadIdx.x & 63;
  int base = 0;
  for (int s0 = 0; s0 < a.S; s0 += kWave) {
    const int sq = s0 + lane;
    const int cnt = sq < a.S ? splits_of(a, sq) : 0;
    int incl = cnt;  // inclusive prefix over the wave
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int o = __shfl_up(incl, off, kWave);
      if (lane >= off) incl += o;
    }
    const int total = __shfl(incl, kWave - 1, kWave);
    if (gs < base + total) {
      const uint64_t past = ballot(base + incl > gs);  // lanes whose prefix passes gs
      const int first = __builtin_ctzll(past);
      s_out = s0 + first;
      first_out = base + __shfl(incl - cnt, first, kWave);
      return;
    }
    base += total;
  }
  s_out = -1;
  first_out = base;
}

typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4_t __attribute__((__vector_size__(4 * sizeof(float))));

// One workgroup per (layer, KV head, sequence, split of kSplitRows retained
// rows); each wave takes a quarter of the split in tiles of 16 rows and keeps
// its own online-softmax state.
//  - S = K_tile Q^T on v_mfma_f32_16x16x32_bf16: A = 16 key rows, B = the
//    group's query heads (16 columns, heads past G are zero). The d axis is
//    permuted so that lane l reads 2D/4 contiguous bytes of row l % 16 (the
//    query uses the same permutation). Lane l then holds head l % 16 for rows
//    4 (l / 16) + 0..3 of the tile.
//  - Softmax per head in that layout: the tile maximum over the four lane
//    groups, a reference per head that moves only when a logit passes it by
//    more than 2^kSlack (so p <= 2^kSlack and rescaling is rare), p = 2^(x - m).
//  - p goes through a per-wave LDS tile to the value lanes: 8 dims of one row
//    per lane (coalesced 16-byte loads), o[g][:] += p[g][row] * v[row][:] in
//    fp32 for the GM heads.
// Waves merge in LDS; decode_combine_kernel merges the splits.
constexpr float kSlack = 16.f;

// Cross-lane exchanges on the vector unit (no LDS round trip): the value of
// lane l ^ 16 and of lane l ^ 32 (gfx950 permlane swaps).
__device__ __forceinline__ float xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  // lanes of even rows get the odd row's value in r[1], lanes of odd rows in r[0]
  return __uint_as_float(((threadIdx.x >> 4) & 1) ? r[0] : r[1]);
}
__device__ __forceinline__ float xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(((threadIdx.x >> 5) & 1) ? r[0] : r[1]);
}
template <int D, int GM>
__global__ __launch_bounds__(kThreads) void decode_mfma_kernel(DecodeArgs a) {
  constexpr int KS = D / 32;          // MFMA k-steps over d
  constexpr int KQ = D / 4;           // d entries per lane group (q = lane / 16) and row
  constexpr int LPR = D / 8;          // value lanes per row (8 dims each)
  constexpr int RPL = kWave / LPR;    // value rows per load instruction
  constexpr int VL = 16 / RPL;        // value loads per lane and tile
  constexpr int NW = kThreads / kWave;
  constexpr int ST = D + 2;           // floats per head in a partial state: o[D], m, z
  static_assert(GM % 4 == 0 && GM <= 16, "heads per group");
  __shared__ __attribute__((aligned(16))) float ptile[NW][16][16];  // p[row][head] per wave
  __shared__ __attribute__((aligned(16))) float fscale[NW][16];     // rescale factors per head
  __shared__ float wstate[NW][GM][ST];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, c16 = lane & 15;
  const int lh = blockIdx.x / a.total_splits;
  const int gs = blockIdx.x - lh * a.total_splits;
  int s, first;
  locate_split(a, gs, s, first);
  s = uniform(s);
  if (s < 0) return;  // past the last split: uniform over the workgroup
  const int j = uniform(gs - first);
  const int l = lh / a.Hkv, h = lh - l * a.Hkv;
  int r0;
  const int R = rows_of(a, s, r0);
  constexpr int kWaveRows = kSplitRows / NW;
  const int w0 = j * kSplitRows + wave * kWaveRows;  // this wave's rows [w0, w1)
  const int w1 = min(R, w0 + kWaveRows);
  // query heads as the B operand: head c16, d = q KQ + 8 ks + 0..7
  bf16x8_t qb[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qb[ks] = bf16x8_t{};
    if (c16 < a.G)
      qb[ks] = *reinterpret_cast<const bf16x8_t*>(
          a.q + (((size_t)l * a.S + s) * a.Hq + h * a.G + c16) * D + q * KQ + 8 * ks);
  }
  const float cl2 = a.scale * 1.44269504088896341f;  // logits in the log2 domain
  float m_ref = -INFINITY;  // reference of head c16 (the same in the four lane groups)
  float zp = 0.f;           // this lane's share of head c16's sum
  float o[GM][8];
#pragma unroll
  for (int g = 0; g < GM; ++g)
#pragma unroll
    for (int i = 0; i < 8; ++i) o[g][i] = 0.f;
  const uint16_t* kb = a.k + ((size_t)lh * a.out_rows + r0) * D;
  const uint16_t* vb = a.v + ((size_t)lh * a.out_rows + r0) * D;
  const int vrow = lane / LPR, vcol = 8 * (lane % LPR);
  // the tile at row t: K as the MFMA A operand, V as 8 dims of a row per lane;
  // rows past the end re-read the last one
  auto load = [&](int t, bf16x8_t (&ka)[KS], u32x4_t (&vw)[VL]) __attribute__((always_inline)) {
    const int rk = min(t + c16, w1 - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      ka[ks] = __builtin_nontemporal_load(
          reinterpret_cast<const bf16x8_t*>(kb + (size_t)rk * D + q * KQ + 8 * ks));
#pragma unroll
    for (int i = 0; i < VL; ++i) {
      const int rv = min(t + i * RPL + vrow, w1 - 1);
      vw[i] = __builtin_nontemporal_load(
          reinterpret_cast<const u32x4_t*>(vb + (size_t)rv * D + vcol));
    }
  };
  for (int t = w0; t < w1; t += 16) {  // wave-uniform loop
    bf16x8_t ka[KS];
    u32x4_t vw[VL];
    load(t, ka, vw);
    // every load of the tile is in flight before the first wait (one memory
    // round trip per tile, not one for K and another for V)
    __builtin_amdgcn_sched_barrier(0);
    f32x4_t acc = f32x4_t{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[ks], qb[ks], acc, 0, 0, 0);
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = t + 4 * q + i < w1 ? acc[i] * cl2 : -INFINITY;
    float tmax = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    // -inf never moves the reference; the first finite tile does
    if (__builtin_amdgcn_ballot_w64(tmax > m_ref + kSlack) != 0) {  // wave-uniform, rare
      // the tile maximum of each head over its four lane groups
      tmax = fmaxf(tmax, xor16(tmax));
      tmax = fmaxf(tmax, xor32(tmax));
      const bool move = tmax > m_ref + kSlack;  // the same in the four lane groups of a head
      const float m_new = move ? tmax : m_ref;
      const float f = m_ref == -INFINITY ? 0.f : fast_exp2(m_ref - m_new);
      zp *= f;
      m_ref = m_new;
      if (q == 0) fscale[wave][c16] = f;
      __builtin_amdgcn_wave_barrier();
      float fs[GM];
#pragma unroll
      for (int g = 0; g < GM; g += 4) {
        const float4 v4 = *reinterpret_cast<const float4*>(&fscale[wave][g]);
        fs[g] = v4.x;
        fs[g + 1] = v4.y;
        fs[g + 2] = v4.z;
        fs[g + 3] = v4.w;
      }
#pragma unroll
      for (int g = 0; g < GM; ++g)
#pragma unroll
        for (int i = 0; i < 8; ++i) o[g][i] *= fs[g];
    }
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p[i] = x[i] == -INFINITY ? 0.f : fast_exp2(x[i] - m_ref);
      zp += p[i];
      ptile[wave][4 * q + i][c16] = p[i];
    }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int i = 0; i < VL; ++i) {
      const int rr = i * RPL + vrow;  // row of the tile
      float pr[GM];
#pragma unroll
      for (int g = 0; g < GM; g += 4) {
        const float4 v4 = *reinterpret_cast<const float4*>(&ptile[wave][rr][g]);
        pr[g] = v4.x;
        pr[g + 1] = v4.y;
        pr[g + 2] = v4.z;
        pr[g + 3] = v4.w;
      }
      float v[8];
      unpack8(vw[i], v);
#pragma unroll
      for (int g = 0; g < GM; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) o[g][e] = fmaf(pr[g], v[e], o[g][e]);
    }
    __builtin_amdgcn_wave_barrier();  // the tile's p reads precede the next tile's writes
  }
  // this wave's sums: z over the four lane groups, o over the row groups of the value lanes
  zp += xor16(zp);
  zp += xor32(zp);
#pragma unroll
  for (int off = LPR; off < kWave; off <<= 1)
#pragma unroll
    for (int g = 0; g < GM; ++g)
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] += __shfl_xor(o[g][i], off, kWave);
  if (lane < LPR) {
#pragma unroll
    for (int g = 0; g < GM; ++g) {
      if (g >= a.G) break;
#pragma unroll
      for (int i = 0; i < 8; ++i) wstate[wave][g][vcol + i] = o[g][i];
    }
  }
  if (q == 0 && c16 < a.G) {
    wstate[wave][c16][D] = m_ref;
    wstate[wave][c16][D + 1] = zp;
  }
  __syncthreads();
  // merge the waves: thread (g, d) for every head g and dim d
  for (int e = tid; e < a.G * D; e += kThreads) {
    const int g = e / D, dd = e - g * D;
    float M = -INFINITY, Z = 0.f, O = 0.f;
    for (int w = 0; w < NW; ++w) {
      const float mw = wstate[w][g][D], zw = wstate[w][g][D + 1];
      const float mn = fmaxf(M, mw);
      if (mn == -INFINITY) continue;
      const float x = fast_exp2(M - mn), y = fast_exp2(mw - mn);
      Z = Z * x + zw * y;
      O = O * x + wstate[w][g][dd] * y;
      M = mn;
    }
    float* part = a.partial + (((size_t)lh * a.total_splits + gs) * a.G + g) * ST;
    part[dd] = O;
    if (dd == 0) {
      part[D] = M;
      part[D + 1] = Z;
    }
  }
}

// out[l][s][hq] = merge of the splits of sequence s (o / z; zero rows give 0).
template <int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(DecodeArgs a) {
  constexpr int ST = D + 2;
  const int hq = blockIdx.x % a.Hq;
  const int s = (blockIdx.x / a.Hq) % a.S;
  const int l = blockIdx.x / (a.Hq * a.S);
  const int lh = l * a.Hkv + hq / a.G, g = hq % a.G;
  const int dd = threadIdx.x;
  if (blockIdx.x == 0 && dd == 0 && a.status && a.cu_retained[a.S] > a.out_rows)
    atomicOr(a.status, kFlagOutRows);  // the split kernel read no row past out_rows
  // global splits of the sequences before s: a wave-wide prefix over 64 sequences at a time
  int first = 0;
  {
    const int lane = dd & 63;
    for (int s0 = 0; s0 < s; s0 += kWave) {
      const int sq = s0 + lane;
      int cnt = sq < s ? splits_of(a, sq) : 0;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off, kWave);
      first += cnt;
    }
  }
  first = min(first, a.total_splits);  // the splits the grid held
  const int last = min(first + splits_of(a, s), a.total_splits);
  float M = -INFINITY, Z = 0.f, O = 0.f;
  for (int g0 = first; g0 < last; g0 += 8) {  // eight splits' loads in flight at a time
    float mw[8], zw[8], ow[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      mw[u] = -INFINITY;
      zw[u] = 0.f;
      ow[u] = 0.f;
      if (g0 + u < last) {
        const float* part = a.partial + (((size_t)lh * a.total_splits + g0 + u) * a.G + g) * ST;
        mw[u] = part[D];
        zw[u] = part[D + 1];
        ow[u] = part[dd];
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float mn = fmaxf(M, mw[u]);
      if (mn == -INFINITY) continue;
      const float x = fast_exp2(M - mn), y = fast_exp2(mw[u] - mn);
      Z = Z * x + zw[u] * y;
      O = O * x + ow[u] * y;
      M = mn;
    }
  }
  a.out[(((size_t)l * a.S + s) * a.Hq + hq) * D + dd] = Z > 0.f ? O / Z : 0.f;
}

}  // namespace

// A bound of sum_s ceil(R_s / kSplitRows) from what the host knows: R_s <=
// min(N_s, out_rows), and sum_s R_s <= out_rows gives at most
// floor(out_rows / kSplitRows) + S splits.
int decode_total_splits(const int32_t* cu_seqlens_host, int S, int out_rows) {
  int64_t acc = 0;
  for (int s = 0; s < S; ++s) {
    const int n = std::min(cu_seqlens_host[s + 1] - cu_seqlens_host[s], out_rows);
    acc += (n + kSplitRows - 1) / kSplitRows;
  }
  return (int)std::min<int64_t>(acc, (int64_t)(out_rows / kSplitRows) + S);
}

size_t decode_partial_floats(const DecodeArgs& a) {
  if (a.G > 16) return 0;
  return (size_t)a.L * a.Hkv * a.total_splits * a.G * (a.d + 2);
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t st) {
  if (a.G > 16) {  // wide query groups: one workgroup per query head
    const dim3 grid((unsigned)(a.L * a.S * a.Hq));
    if (a.d == 128)
      hipLaunchKernelGGL(decode_simple_kernel<128>, grid, dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL(decode_simple_kernel<64>, grid, dim3(kThreads), 0, st, a);
    return hipGetLastError();
  }
  if (a.total_splits > 0) {
    const dim3 grid((unsigned)(a.L * a.Hkv) * (unsigned)a.total_splits);
    auto go = [&](auto d_c, auto gm_c) {
      constexpr int Dd = decltype(d_c)::value, GMm = decltype(gm_c)::value;
      hipLaunchKernelGGL((decode_mfma_kernel<Dd, GMm>), grid, dim3(kThreads), 0, st, a);
    };
    using I128 = std::integral_constant<int, 128>;
    using I64 = std::integral_constant<int, 64>;
    using G4 = std::integral_constant<int, 4>;
    using G8 = std::integral_constant<int, 8>;
    using G16 = std::integral_constant<int, 16>;
    if (a.d == 128) {
      if (a.G <= 4) go(I128{}, G4{});
      else if (a.G <= 8) go(I128{}, G8{});
      else go(I128{}, G16{});
    } else {
      if (a.G <= 4) go(I64{}, G4{});
      else if (a.G <= 8) go(I64{}, G8{});
      else go(I64{}, G16{});
    }
  }
  const dim3 cgrid((unsigned)(a.L * a.S * a.Hq));
  if (a.d == 128)
    hipLaunchKernelGGL(decode_combine_kernel<128>, cgrid, dim3(128), 0, st, a);
  else
    hipLaunchKernelGGL(decode_combine_kernel<64>, cgrid, dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace stepkv
