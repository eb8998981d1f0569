// One decode step over the compacted cache C_hat: out = softmax(scale *
// q . K_hat^T) V_hat for every (layer, sequence, query head), fp32
// accumulation (the consumer of the compacted cache, Sec. 3).
//
// decode_split_kernel: one workgroup per (layer, KV head, sequence, split of
// 512 retained rows) serves all G query heads of the KV head, so K and V are
// read once. 16-byte pieces, 2d/16 lanes per row (coalesced rows), the next
// four rows' loads issued before the current four rows' arithmetic; q . k from
// the raw bf16 pairs (v_dot2 with fp32 sums, scale applied after), an exact
// online softmax per head in the log2 domain; a row's lanes sum by DPP, lane
// groups merge by shuffles, waves in LDS, and decode_combine_kernel merges the
// splits. decode_simple_kernel serves groups wider than 8 query heads.
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


#ifndef STEPKV_DECODE_SPLIT_ROWS
#define STEPKV_DECODE_SPLIT_ROWS 512
#endif
constexpr int kSplitRows = STEPKV_DECODE_SPLIT_ROWS;  // retained rows per workgroup

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16x2_t as_bf16x2(unsigned int w) {
  return __builtin_bit_cast(bf16x2_t, w);
}

__device__ __forceinline__ void unpack8(const u32x4_t& w, float (&f)[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

// Sum over the LPR lanes of a row (8 or 16 consecutive lanes, one DPP row or
// half-row) with DPP lane permutes: swap neighbours, swap pairs, mirror the
// half-row, mirror the row. Every lane of the group ends with the sum.
template <int LPR>
__device__ __forceinline__ float row_sum(float v) {
  static_assert(LPR == 8 || LPR == 16, "lanes per row");
  auto dpp = [](float x, auto ctrl_c) __attribute__((always_inline)) {
    constexpr int ctrl = decltype(ctrl_c)::value;
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), ctrl, 0xf, 0xf, false));
  };
  v += dpp(v, std::integral_constant<int, 0xb1>{});   // quad_perm [1,0,3,2]
  v += dpp(v, std::integral_constant<int, 0x4e>{});   // quad_perm [2,3,0,1]
  v += dpp(v, std::integral_constant<int, 0x141>{});  // row_half_mirror
  if constexpr (LPR == 16) v += dpp(v, std::integral_constant<int, 0x140>{});  // row_mirror
  return v;
}

// Merge online-softmax state (m, z, o) with another (log2 domain).
template <int N>
__device__ __forceinline__ void merge_state(float& m, float& z, float (&o)[N], float mo, float zo,
                                            const float (&oo)[N]) {
  const float mn = fmaxf(m, mo);
  if (mn == -INFINITY) return;  // both empty
  const float a = fast_exp2(m - mn), b = fast_exp2(mo - mn);
  z = z * a + zo * b;
#pragma unroll
  for (int i = 0; i < N; ++i) o[i] = o[i] * a + oo[i] * b;
  m = mn;
}

// Row splits of sequence s: ceil(min(N_s, out_rows) / kSplitRows).
__device__ __forceinline__ int splits_of(const DecodeArgs& a, int s) {
  const int n = min(a.cu_seqlens[s + 1] - a.cu_seqlens[s], a.out_rows);
  return (n + kSplitRows - 1) / kSplitRows;
}

// The sequence holding global split gs, and the first global split of that
// sequence: a wave-wide prefix sum over 64 sequences at a time.
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
  s_out = a.S - 1;  // not reached for gs < total_splits
  first_out = base;
}

template <int D, int GM>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(DecodeArgs a) {
  constexpr int LPR = 2 * D / 16;        // lanes per 2d-byte row
  constexpr int GPW = kWave / LPR;       // row groups per wave
  constexpr int NG = (kThreads / kWave) * GPW;
  constexpr int ST = D + 2;              // floats per head in a partial state: o[D], m, z
  __shared__ float wstate[kThreads / kWave][GM][ST];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane % LPR, grp = wave * GPW + lane / LPR;
  const int lh = blockIdx.x / a.total_splits;
  const int gs = blockIdx.x - lh * a.total_splits;
  int s, first;
  locate_split(a, gs, s, first);
  s = uniform(s);
  const int j = uniform(gs - first);
  const int l = lh / a.Hkv, h = lh - l * a.Hkv;
  const int r0 = a.cu_retained[s];
  const int R = max(0, min(a.cu_retained[s + 1], a.out_rows) - r0);
  const int row_end = min(R, (j + 1) * kSplitRows);
  // this lane's 8 dims (4 bf16 pairs) of every query head of the group
  u32x4_t q[GM];
  const float qs = a.scale * 1.44269504088896341f;  // logits in the log2 domain
#pragma unroll
  for (int g = 0; g < GM; ++g) {
    q[g] = u32x4_t{0u, 0u, 0u, 0u};
    if (g < a.G)
      q[g] = *reinterpret_cast<const u32x4_t*>(
          a.q + (((size_t)l * a.S + s) * a.Hq + h * a.G + g) * D + 8 * sub);
  }
  float m[GM], z[GM], o[GM][8];
#pragma unroll
  for (int g = 0; g < GM; ++g) {
    m[g] = -INFINITY;
    z[g] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[g][i] = 0.f;
  }
  const u32x4_t* kb = reinterpret_cast<const u32x4_t*>(a.k + ((size_t)lh * a.out_rows + r0) * D);
  const u32x4_t* vb = reinterpret_cast<const u32x4_t*>(a.v + ((size_t)lh * a.out_rows + r0) * D);
  // one online-softmax update for NR rows r, r + NG, ...; rows at or past
  // row_end re-read the first row and count as absent
  constexpr int NR = 4;
  auto update = [&](const u32x4_t (&kw)[NR], const u32x4_t (&vw)[NR], int r)
      __attribute__((always_inline)) {
    float v[NR][8];
#pragma unroll
    for (int b = 0; b < NR; ++b) unpack8(vw[b], v[b]);
#pragma unroll
    for (int g = 0; g < GM; ++g) {
      if (g >= a.G) break;
      float dt[NR];
#pragma unroll
      for (int b = 0; b < NR; ++b) {
        float acc = 0.f;  // exact bf16 products, fp32 sums
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q[g][i]), as_bf16x2(kw[b][i]), acc,
                                                false);
        dt[b] = r + b * NG < row_end ? row_sum<LPR>(acc) * qs : -INFINITY;
      }
      float mn = m[g];
#pragma unroll
      for (int b = 0; b < NR; ++b) mn = fmaxf(mn, dt[b]);
      const float sc = fast_exp2(m[g] - mn);
      float p[NR], zs = 0.f;
#pragma unroll
      for (int b = 0; b < NR; ++b) {
        p[b] = fast_exp2(dt[b] - mn);
        zs += p[b];
      }
      z[g] = fmaf(z[g], sc, zs);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float t = p[0] * v[0][i];
#pragma unroll
        for (int b = 1; b < NR; ++b) t = fmaf(p[b], v[b][i], t);
        o[g][i] = fmaf(o[g][i], sc, t);
      }
      m[g] = mn;
    }
  };
  auto load = [&](int rr, u32x4_t (&kw)[NR], u32x4_t (&vw)[NR]) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < NR; ++b) {
      const int ri = rr + b * NG < row_end ? rr + b * NG : rr;
      kw[b] = __builtin_nontemporal_load(kb + (size_t)ri * LPR + sub);
      vw[b] = __builtin_nontemporal_load(vb + (size_t)ri * LPR + sub);
    }
  };
  int r = j * kSplitRows + grp;
  u32x4_t ck[NR], cv[NR];
  if (r < row_end) load(r, ck, cv);
  while (r < row_end) {  // the next rows' loads go out before this batch's arithmetic
    const int rn = r + NR * NG;
    u32x4_t nk[NR], nv[NR];
    if (rn < row_end) load(rn, nk, nv);
    update(ck, cv, r);
#pragma unroll
    for (int b = 0; b < NR; ++b) {
      ck[b] = nk[b];
      cv[b] = nv[b];
    }
    r = rn;
  }
  // merge the row groups of this wave (lanes with the same piece)
#pragma unroll
  for (int off = LPR; off < kWave; off <<= 1) {
#pragma unroll
    for (int g = 0; g < GM; ++g) {
      if (g >= a.G) break;
      float oo[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) oo[i] = __shfl_xor(o[g][i], off, kWave);
      const float mo = __shfl_xor(m[g], off, kWave), zo = __shfl_xor(z[g], off, kWave);
      merge_state(m[g], z[g], o[g], mo, zo, oo);
    }
  }
  if (lane < LPR) {
#pragma unroll
    for (int g = 0; g < GM; ++g) {
      if (g >= a.G) break;
#pragma unroll
      for (int i = 0; i < 8; ++i) wstate[wave][g][8 * sub + i] = o[g][i];
      if (sub == 0) {
        wstate[wave][g][D] = m[g];
        wstate[wave][g][D + 1] = z[g];
      }
    }
  }
  __syncthreads();
  // merge the waves: thread (g, d) for every head g and dim d
  for (int e = tid; e < a.G * D; e += kThreads) {
    const int g = e / D, dd = e - g * D;
    float M = -INFINITY, Z = 0.f, O = 0.f;
    for (int w = 0; w < kThreads / kWave; ++w) {
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
  int first = 0;  // global splits of the sequences before s (every lane adds them all)
  for (int s2 = 0; s2 < s; ++s2) first += splits_of(a, s2);
  const int last = first + splits_of(a, s);
  float M = -INFINITY, Z = 0.f, O = 0.f;
  for (int gs = first; gs < last; ++gs) {
    const float* part = a.partial + (((size_t)lh * a.total_splits + gs) * a.G + g) * ST;
    const float mw = part[D], zw = part[D + 1];
    const float mn = fmaxf(M, mw);
    if (mn == -INFINITY) continue;
    const float x = fast_exp2(M - mn), y = fast_exp2(mw - mn);
    Z = Z * x + zw * y;
    O = O * x + part[dd] * y;
    M = mn;
  }
  a.out[(((size_t)l * a.S + s) * a.Hq + hq) * D + dd] = Z > 0.f ? O / Z : 0.f;
}

}  // namespace

int decode_total_splits(const int32_t* cu_seqlens_host, int S, int out_rows) {
  int acc = 0;
  for (int s = 0; s < S; ++s) {
    const int n = std::min(cu_seqlens_host[s + 1] - cu_seqlens_host[s], out_rows);
    acc += (n + kSplitRows - 1) / kSplitRows;
  }
  return acc;
}

size_t decode_partial_floats(const DecodeArgs& a) {
  if (a.G > 8) return 0;
  return (size_t)a.L * a.Hkv * a.total_splits * a.G * (a.d + 2);
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t st) {
  if (a.G > 8) {  // wide query groups: one workgroup per query head
    const dim3 grid((unsigned)(a.L * a.S * a.Hq));
    if (a.d == 128)
      hipLaunchKernelGGL(decode_simple_kernel<128>, grid, dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL(decode_simple_kernel<64>, grid, dim3(kThreads), 0, st, a);
    return hipGetLastError();
  }
  if (a.total_splits > 0) {
    const dim3 grid((unsigned)(a.L * a.Hkv) * (unsigned)a.total_splits);
    if (a.d == 128) {
      if (a.G <= 4) hipLaunchKernelGGL((decode_split_kernel<128, 4>), grid, dim3(kThreads), 0, st, a);
      else hipLaunchKernelGGL((decode_split_kernel<128, 8>), grid, dim3(kThreads), 0, st, a);
    } else {
      if (a.G <= 4) hipLaunchKernelGGL((decode_split_kernel<64, 4>), grid, dim3(kThreads), 0, st, a);
      else hipLaunchKernelGGL((decode_split_kernel<64, 8>), grid, dim3(kThreads), 0, st, a);
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
