// One decode step over the compacted cache C_hat: out = softmax(scale *
// q . K_hat^T) V_hat for every (layer, sequence, query head), fp32
// accumulation (the consumer of the compacted cache, Sec. 3).
//
// decode_mfma_kernel: one workgroup per (layer, KV head, sequence, split of
// 512 or 1024 retained rows) serves all G <= 16 query heads of the KV head, so K and V
// are read once: q . k and p V for the whole query group on MFMA with an
// exact online softmax per head between them, several 16-row tiles in flight
// per wave; decode_combine_kernel merges the splits. decode_simple_kernel
// serves groups wider than 16 heads.
#include "common.h"
#include "internal.h"

#include <math.h>

#include <algorithm>
#include <type_traits>
#include <utility>

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

// Row splits of sequence s: ceil(R_s / split_rows).
__device__ __forceinline__ int splits_of(const DecodeArgs& a, int s) {
  int r0;
  return (rows_of(a, s, r0) + a.split_rows - 1) / a.split_rows;
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

// One workgroup per (layer, KV head, sequence, split of split_rows retained
// rows); each wave takes a quarter of the split in tiles of 16 rows, keeps its
// own online-softmax state and its own ring of kStages tiles: K to registers,
// V straight to LDS (global_load_lds), tile t + kStages - 1 issued before
// tile t is computed. Both products run on MFMA with the query group as
// 16 columns (heads past G are zero):
//  - S = K_tile Q^T on v_mfma_f32_16x16x32_bf16: A = the 16 key rows, B = the
//    query heads. Lane group g = l / 16 reads 16-byte pieces 4 ks + g of its
//    row for k-step ks (64 contiguous bytes per row and load; the query takes
//    the same d order). Lane l then holds head l % 16 for rows 4 g + 0..3.
//  - Softmax per head in that layout, in the log2 domain: a reference m per
//    head that moves only when a logit exceeds it by more than kSlack (so
//    p = 2^(x - m) <= 2^kSlack and rescaling is rare).
//  - O += P V on v_mfma_f32_16x16x16_bf16: A = P as the lanes hold it (head
//    l % 16, rows 4 g + 0..3), split into bf16 hi + lo parts (P to about
//    2^-17 relative); B = 16 value columns of those rows, read from the LDS
//    tile with the transposing read ds_read_b64_tr_b16. Lane l then holds
//    heads 4 g + 0..3 of the 16 columns.
// The V tile in LDS is row-major with the 32-byte pairs of row r XOR-swizzled
// by swz(r), so that the 32 lanes of each transposing read hit distinct banks.
// Waves merge in LDS; decode_combine_kernel merges the splits.
constexpr float kSlack = 16.f;

// Tiles per wave in the ring: one computed while the next is in flight (a
// deeper ring costs occupancy and measured no faster).
constexpr int kStages = 2;

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

typedef short i16x4_t __attribute__((ext_vector_type(4)));

// f(integral_constant<int, 0>) ... f(integral_constant<int, N - 1>), unrolled.
template <typename F, int... U>
__device__ __forceinline__ void static_for_impl(F& f, std::integer_sequence<int, U...>) {
  (f(std::integral_constant<int, U>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// XOR swizzle (in 32-byte pairs) of row r of a V tile: rows 8k .. 8k + 7 land
// on distinct bank groups (D = 128: 8 pairs a row; D = 64: 4 pairs a row, two
// rows per 256 bytes).
template <int D>
__device__ __forceinline__ int swz(int r) {
  return D == 128 ? (r & 7) : ((r >> 1) & 3);
}

// Transposing LDS read at byte address addr + OFF. Issued as assembly so that
// the compiler, which cannot tell the ring slots apart, puts no wait for the
// whole ring's direct-to-LDS loads in front of it; completion is awaited with
// tr_settle.
template <int OFF>
__device__ __forceinline__ i16x4_t lds_read_tr(uint32_t addr) {
  i16x4_t v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF) : "memory");
  return v;
}

template <int N>
__device__ __forceinline__ void tr_settle(i16x4_t (&f)[N]) {
  static_assert(N == 4 || N == 8, "value blocks");
  if constexpr (N == 4) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]));
  } else {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]), "+v"(f[5]),
                   "+v"(f[6]), "+v"(f[7]));
  }
}

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3)))
void decode_mfma_kernel(DecodeArgs a) {
  constexpr int KS = D / 32;         // 16-byte K pieces per lane and row = S k-steps
  constexpr int PR = D / 8;          // 16-byte pieces per row
  constexpr int RPI = kWave / PR;    // V rows per direct-to-LDS load
  constexpr int VL = 16 / RPI;       // V loads per tile
  constexpr int NLD = KS + VL;       // vector memory operations per tile and lane
  constexpr int NB = D / 16;         // 16-column blocks of O
  constexpr int NW = kThreads / kWave;
  constexpr int ST = D + 2;          // floats per head in a partial state: o[D], m, z
  constexpr int TB = 16 * D * 2;     // bytes of a V tile
  constexpr int kRingBytes = NW * kStages * TB, kStateBytes = NW * 16 * ST * 4;
  // the V rings during the sweep; the per-wave states [NW][16][ST] after it
  __shared__ __attribute__((aligned(16)))
  uint8_t smem[kRingBytes > kStateBytes ? kRingBytes : kStateBytes];
  __shared__ __attribute__((aligned(16))) float fscale[NW][16];  // rescale factors
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int g4 = lane >> 4, c16 = lane & 15;
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
  const int wave_rows = a.split_rows / NW;
  const int w0 = j * a.split_rows + wave * wave_rows;  // this wave's rows [w0, w1)
  const int w1 = min(R, w0 + wave_rows);
  const int ntiles = w1 > w0 ? (w1 - w0 + 15) / 16 : 0;
  // query heads as the B operand of S: head c16, d piece 4 ks + g4
  bf16x8_t qb[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qb[ks] = bf16x8_t{};
    if (c16 < a.G)
      qb[ks] = *reinterpret_cast<const bf16x8_t*>(
          a.q + (((size_t)l * a.S + s) * a.Hq + h * a.G + c16) * D + 8 * (4 * ks + g4));
  }
  const float cl2 = a.scale * 1.44269504088896341f;  // logits in the log2 domain
  float m_ref = -INFINITY;  // reference of head c16 (the same in the four lane groups)
  float zp = 0.f;           // this lane's share of head c16's sum
  f32x4_t o[NB];            // O[head 4 g4 + i][16 nb + c16]
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) o[nb] = f32x4_t{};
  const uint16_t* kb = a.k + ((size_t)lh * a.out_rows + r0) * D;
  const uint16_t* vb = a.v + ((size_t)lh * a.out_rows + r0) * D;
  uint8_t* ring = smem + wave * (kStages * TB);  // this wave's V tiles
  // direct-to-LDS loads: lane l fills LDS piece l % PR of row i RPI + l / PR,
  // which holds global piece (l % PR) ^ 2 swz(row)
  const int vrow = lane / PR;
  const int vpiece = lane % PR;
  // transposing reads: lane (g4, c16) supplies row 4 g4 + c16 / 4, columns
  // 16 nb + 4 (c16 % 4) .. + 3 (8 bytes of pair nb ^ swz(row))
  uint32_t tr_addr[NB];
  {
    const int r = 4 * g4 + (c16 >> 2);
    const uint32_t base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(
                              (__attribute__((address_space(3))) uint8_t*)ring)) +
                          r * (2 * D) + 8 * (c16 & 3);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) tr_addr[nb] = base + 32 * (nb ^ swz<D>(r));
  }
  bf16x8_t ka[kStages][KS];
  auto issue = [&](int tt, auto slot_c) __attribute__((always_inline)) {
    constexpr int slot = decltype(slot_c)::value;
    const int t = w0 + 16 * tt;
    const int rk = min(t + c16, w1 - 1);  // rows past the end re-read the last one
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      ka[slot][ks] = __builtin_nontemporal_load(
          reinterpret_cast<const bf16x8_t*>(kb + (size_t)rk * D + 8 * (4 * ks + g4)));
#pragma unroll
    for (int i = 0; i < VL; ++i) {
      const int r = i * RPI + vrow;
      const int rv = min(t + r, w1 - 1);
      __builtin_amdgcn_global_load_lds(
          static_cast<const void*>(vb + (size_t)rv * D + 8 * (vpiece ^ (2 * swz<D>(r)))),
          (__attribute__((address_space(3))) void*)(ring + slot * TB + i * (16 * kWave)), 16, 0,
          2);  // non-temporal, like the K loads: every row is read once
    }
  };
  auto compute = [&](int tt, auto slot_c) __attribute__((always_inline)) {
    constexpr int slot = decltype(slot_c)::value;
    const int t = w0 + 16 * tt;
    wait_tiles<NLD, kStages - 1>(min(kStages - 1, ntiles - 1 - tt));
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) settle(ka[slot][ks]);
    // V blocks of this tile from LDS while S runs on the matrix cores
    i16x4_t vbop[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) vbop[nb] = lds_read_tr<slot * TB>(tr_addr[nb]);
    f32x4_t acc = f32x4_t{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[slot][ks], qb[ks], acc, 0, 0, 0);
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = t + 4 * g4 + i < w1 ? acc[i] * cl2 : -INFINITY;
    float tmax = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    // -inf never moves the reference; the first finite tile does
    if (__builtin_amdgcn_ballot_w64(tmax > m_ref + kSlack) != 0) {  // wave-uniform, rare
      tmax = fmaxf(tmax, xor16(tmax));  // the tile maximum of each head
      tmax = fmaxf(tmax, xor32(tmax));
      const bool move = tmax > m_ref + kSlack;  // the same in the four lane groups of a head
      const float m_new = move ? tmax : m_ref;
      const float f = m_ref == -INFINITY ? 0.f : fast_exp2(m_ref - m_new);
      zp *= f;
      m_ref = m_new;
      if (g4 == 0) fscale[wave][c16] = f;
      __builtin_amdgcn_wave_barrier();
      const float4 f4 = *reinterpret_cast<const float4*>(&fscale[wave][4 * g4]);  // heads 4 g4 + i
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        o[nb][0] *= f4.x;
        o[nb][1] *= f4.y;
        o[nb][2] *= f4.z;
        o[nb][3] *= f4.w;
      }
    }
    i16x4_t ph, pl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float pi = x[i] == -INFINITY ? 0.f : fast_exp2(x[i] - m_ref);
      zp += pi;
      const __bf16 hi = (__bf16)pi;
      ph[i] = __builtin_bit_cast(short, hi);
      pl[i] = __builtin_bit_cast(short, (__bf16)(pi - (float)hi));
    }
    tr_settle(vbop);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      o[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ph, vbop[nb], o[nb], 0, 0, 0);
      o[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pl, vbop[nb], o[nb], 0, 0, 0);
    }
  };
  // the ring: tiles 0 .. kStages - 2 first, then tile tt + kStages - 1 (into
  // the slot tile tt - 1 left) before tile tt is computed
  static_for<kStages - 1>([&](auto u_c) __attribute__((always_inline)) {
    if (decltype(u_c)::value < ntiles) issue(decltype(u_c)::value, u_c);
  });
  for (int t0 = 0; t0 < ntiles; t0 += kStages) {  // wave-uniform loop
    static_for<kStages>([&](auto u_c) __attribute__((always_inline)) {
      constexpr int u = decltype(u_c)::value;
      const int tt = t0 + u;
      if (tt >= ntiles) return;
      if (tt + kStages - 1 < ntiles)
        issue(tt + kStages - 1, std::integral_constant<int, (u + kStages - 1) % kStages>{});
      compute(tt, u_c);
    });
  }
  // this wave's sums: z over the four lane groups of each head
  zp += xor16(zp);
  zp += xor32(zp);
  __syncthreads();  // the states overwrite the V rings of every wave
  auto wstate = reinterpret_cast<float(*)[16][ST]>(smem);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (4 * g4 + i < a.G) wstate[wave][4 * g4 + i][16 * nb + c16] = o[nb][i];
  if (g4 == 0 && c16 < a.G) {
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
      const float xa = fast_exp2(M - mn), ya = fast_exp2(mw - mn);
      Z = Z * xa + zw * ya;
      O = O * xa + wstate[w][g][dd] * ya;
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

// 1024 rows per split when the cache fills the chip's resident workgroups
// (256 CUs x 3) at least twice over with them, else 512: longer splits spend
// less of each workgroup's life on its start and merge, shorter ones keep a
// small cache spread over every CU.
int decode_split_rows(int L, int Hkv, int out_rows) {
  constexpr int64_t kResident = 256 * 3;
  return (int64_t)L * Hkv * (out_rows / 1024) >= 2 * kResident ? 1024 : 512;
}

// A bound of sum_s ceil(R_s / split_rows) from what the host knows: R_s <=
// min(N_s, out_rows), and sum_s R_s <= out_rows gives at most
// floor(out_rows / split_rows) + S splits.
int decode_total_splits(const int32_t* cu_seqlens_host, int S, int out_rows, int split_rows) {
  int64_t acc = 0;
  for (int s = 0; s < S; ++s) {
    const int n = std::min(cu_seqlens_host[s + 1] - cu_seqlens_host[s], out_rows);
    acc += (n + split_rows - 1) / split_rows;
  }
  return (int)std::min<int64_t>(acc, (int64_t)(out_rows / split_rows) + S);
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
    if (a.d == 128)
      hipLaunchKernelGGL(decode_mfma_kernel<128>, grid, dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL(decode_mfma_kernel<64>, grid, dim3(kThreads), 0, st, a);
  }
  const dim3 cgrid((unsigned)(a.L * a.S * a.Hq));
  if (a.d == 128)
    hipLaunchKernelGGL(decode_combine_kernel<128>, cgrid, dim3(128), 0, st, a);
  else
    hipLaunchKernelGGL(decode_combine_kernel<64>, cgrid, dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace stepkv
