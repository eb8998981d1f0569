// Observation-window token saliency (Sec. 5.2, token saliency T_i):
//   A_i = sum over window rows r of softmax_i(scale * q_r . k_i)
// for every (sequence, layer, KV head), exactly, in two sweeps over K.
//
// The row softmax needs each row's log-sum-exp over all N keys before any
// column can be summed, so the kernel runs
//   pass 1  per key chunk: z = K Q^T on MFMA, per-row running (max, sum exp)
//   combine per row: merge the chunk partials into log2-domain LSE
//   pass 2  per key chunk: z = Q K^T on MFMA, A_i = sum_r exp2(c z - lse_r)
// The two passes swap the MFMA operands so that each reduction stays inside
// a lane: in pass 1 a lane holds 16 keys of one window row, in pass 2 16
// window rows of one key (v_mfma_f32_32x32x16_bf16 output layout).
//
// K tiles stream HBM -> LDS with global_load_lds_dwordx4 (fully coalesced,
// no VGPR round trip) into an XOR-swizzled ring of NBUF buffers; Q stays in
// VGPRs for the whole chunk. One barrier per tile.
#include "common.h"
#include "internal.h"

#include <math.h>

namespace stepkv {
namespace {

constexpr int kThreads = 256;  // 4 waves: (row group) x (key group)

// XOR swizzle of the 16-byte pieces of key row r inside a K tile. The 16 lanes
// of a ds_read_b128 phase read the same logical piece of 16 consecutive rows;
// the swizzle spreads them over 16 distinct 16-byte bank groups (a 256-byte
// row for d = 128; two 128-byte rows per bank line for d = 64).
template <int D>
__device__ __forceinline__ int swizzle(int r) {
  return D == 128 ? (r & 15) : ((r >> 1) & 7);
}

// Byte offset of logical 16-byte piece p of key row r inside a K tile.
template <int D>
__device__ __forceinline__ int tile_offset(int r, int p) {
  return r * (2 * D) + 16 * (p ^ swizzle<D>(r));
}

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

#ifndef STEPKV_SAL_RING_BYTES
#define STEPKV_SAL_RING_BYTES 32768
#endif

// Make the compiler wait for the load that produced x here, once, instead of
// at the first use inside the tile loop, where its wait would also drain the
// K prefetch ring on every iteration.
template <typename T>
__device__ __forceinline__ void settle(T& x) {
  asm volatile("" : "+v"(x));
}

// One 16-byte LDS read of the K ring. Issued as assembly so that the compiler,
// which cannot tell the ring slots apart, does not put a vmcnt(0) (a wait for
// the whole prefetch ring) in front of it; completion is awaited explicitly
// with lds_settle.
__device__ __forceinline__ bf16x8_t lds_read_b128(uint32_t addr) {
  bf16x8_t v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr) : "memory");
  return v;
}

template <int N>
__device__ __forceinline__ void lds_settle(bf16x8_t (&f)[N]) {
  static_assert(N == 4 || N == 8, "fragment count");
  if constexpr (N == 4) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]));
  } else {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]), "+v"(f[5]),
                   "+v"(f[6]), "+v"(f[7]));
  }
}

// LDS writes of this wave complete, then a workgroup barrier. Outstanding
// global loads (the K prefetch ring) are deliberately not waited for.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__global__ void chunk_plan_kernel(const int32_t* __restrict__ cu_seqlens,
                                  int32_t* __restrict__ cu_chunks, int S, int chunk) {
  if (threadIdx.x == 0) {
    int acc = 0;
    cu_chunks[0] = 0;
    for (int s = 0; s < S; ++s) {
      const int n = cu_seqlens[s + 1] - cu_seqlens[s];
      acc += (n + chunk - 1) / chunk;
      cu_chunks[s + 1] = acc;
    }
  }
}

// D: head dim. RG: row groups of 64 window rows (1, 2 or 4); the 4 / RG
// waves per row group split each key tile into 32-key sub-tiles.
template <int D, int RG, int PASS>
__global__ __launch_bounds__(kThreads, 2) void saliency_kernel(SaliencyArgs a) {
  constexpr int KG = 4 / RG;
  constexpr int TILE = 32 * KG;               // keys per workgroup iteration
  constexpr int KSTEPS = D / 16;              // MFMA k-steps
  constexpr int TILE_BYTES = TILE * 2 * D;
  constexpr int NBUF = STEPKV_SAL_RING_BYTES / TILE_BYTES >= 2 ? STEPKV_SAL_RING_BYTES / TILE_BYTES : 2;
  constexpr int NLD = TILE_BYTES / (kThreads * 16);  // 16-byte loads per thread per tile
  static_assert(NLD >= 1, "tile too small");
  __shared__ __attribute__((aligned(16))) uint8_t kbuf[NBUF * TILE_BYTES];
  __shared__ float red[2 * kThreads];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int rg = wave % RG, kg = wave / RG;
  const int col = lane & 31, hf = lane >> 5;

  // ---- work item: (head lh, sequence s, chunk c)
  const int LH = a.L * a.Hkv;
  int lh = blockIdx.x / a.total_chunks;
  const int rem = blockIdx.x - lh * a.total_chunks;
  if (PASS == 2) lh = LH - 1 - lh;  // pass 2 starts where pass 1 ended (cache reuse)
  const int s = segment_of(a.cu_chunks, a.S, rem);
  const int c = rem - a.cu_chunks[s];
  const int l = lh / a.Hkv, h = lh - l * a.Hkv;
  const int seq0 = a.cu_seqlens[s];
  const int ns = a.cu_seqlens[s + 1] - seq0;
  const int key0 = c * a.chunk;
  const int nkeys = min(a.chunk, ns - key0);
  const int ntiles = (nkeys + TILE - 1) / TILE;
  const uint16_t* __restrict__ kseq = a.k + ((size_t)lh * a.ntot + seq0) * D;

  // ---- window rows of this wave: two 32-row blocks, k-slices (D/2)*hf + 8*st
  bf16x8_t qf[2][KSTEPS];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int row = rg * 64 + b * 32 + col;
    if (row < a.R) {
      const int w = row / a.G, g = row - w * a.G;
      const uint16_t* qp =
          a.q + ((((size_t)l * a.S + s) * a.W + w) * a.Hq + h * a.G + g) * D + (D / 2) * hf;
#pragma unroll
      for (int st = 0; st < KSTEPS; ++st)
        qf[b][st] = *reinterpret_cast<const bf16x8_t*>(qp + 8 * st);
    } else {
#pragma unroll
      for (int st = 0; st < KSTEPS; ++st) qf[b][st] = bf16x8_t{};
    }
  }

  const uint32_t kbuf_lds = static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t*)kbuf));
  auto issue_tile = [&](int t) {
    uint8_t* base = kbuf + (t % NBUF) * TILE_BYTES;
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int o = 16 * (tid + kThreads * j);  // this lane's 16 bytes of the tile
      const int r = o / (2 * D);
      const int pp = (o % (2 * D)) / 16;
      const int p = pp ^ swizzle<D>(r);
      const int key = min(key0 + t * TILE + r, ns - 1);  // tail rows re-read a valid key
      const uint16_t* src = kseq + (size_t)key * D + 8 * p;
      uint8_t* dst = base + 16 * (kThreads * j + 64 * wave);  // lane l lands at dst + 16 l
      __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)dst, 16, 0,
                                       0);
    }
  };

  // pass 1 state: per lane, per row block, running log2-domain max and sum
  float m2[2] = {-INFINITY, -INFINITY};
  float zs[2] = {0.f, 0.f};
  // pass 2 state: log2-domain LSE of the 16 rows this lane holds per block
  float lr[2][16];
  if (PASS == 2) {
    const float* lp = a.lse2 + ((size_t)s * LH + lh) * a.rows_pad + rg * 64;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int j = 0; j < 16; ++j) lr[b][j] = lp[b * 32 + 8 * (j >> 2) + 4 * hf + (j & 3)];
  }

#pragma unroll
  for (int b = 0; b < 2; ++b) {
#pragma unroll
    for (int st = 0; st < KSTEPS; ++st) settle(qf[b][st]);
    if (PASS == 2) {
#pragma unroll
      for (int j = 0; j < 16; ++j) settle(lr[b][j]);
    }
  }

  auto reduce_tile = [&](int t) {  // pass 2: sum the per-wave column partials of tile t
    if (tid < TILE) {
      const int kg2 = tid >> 5, col2 = tid & 31;
      const float* rp = red + (t & 1) * kThreads;
      float sum = 0.f;
#pragma unroll
      for (int r2 = 0; r2 < RG; ++r2) {
        const int w2 = kg2 * RG + r2;
        sum += rp[w2 * 64 + col2];
        sum += rp[w2 * 64 + 32 + col2];
      }
      const int key = t * TILE + tid;
      if (key < nkeys) a.sal[(size_t)lh * a.ntot + seq0 + key0 + key] = sum;
    }
  };

  const int kr = kg * 32 + col;
  auto read_frags = [&](int t, bf16x8_t(&kf)[KSTEPS]) {
    const uint32_t tb = kbuf_lds + (t % NBUF) * TILE_BYTES;
#pragma unroll
    for (int st = 0; st < KSTEPS; ++st)
      kf[st] = lds_read_b128(tb + tile_offset<D>(kr, (D / 16) * hf + st));
    lds_settle(kf);
  };
  auto mfma_tile = [&](const bf16x8_t(&kf)[KSTEPS], f32x16_t(&acc)[2]) {
    acc[0] = f32x16_t{};
    acc[1] = f32x16_t{};
#pragma unroll
    for (int st = 0; st < KSTEPS; ++st) {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        if (PASS == 1)
          acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st], qf[b][st], acc[b], 0, 0, 0);
        else
          acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[b][st], kf[st], acc[b], 0, 0, 0);
      }
    }
  };
  // Softmax work on a finished tile t. Only the last tile can be partial.
  auto finish_tile = [&](const f32x16_t(&acc)[2], int t, bool full) {
    if (PASS == 1) {
      // lane: window row `col` of block b; keys t*TILE + kg*32 + 8*(j/4) + 4*hf + (j%4)
      const int kbase = t * TILE + kg * 32 + 4 * hf;
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        float v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          v[j] = acc[b][j];
          if (!full && kbase + 8 * (j >> 2) + (j & 3) >= nkeys) v[j] = -INFINITY;
        }
        float tmax = v[0];
#pragma unroll
        for (int j = 1; j < 16; ++j) tmax = fmaxf(tmax, v[j]);
        const float mnew = fmaxf(m2[b], tmax * a.c);
        const float f = fast_exp2(m2[b] - mnew);  // rescale of the running sum
        float p4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 16; ++j) p4[j & 3] += fast_exp2(fmaf(v[j], a.c, -mnew));
        const float sum = (p4[0] + p4[1]) + (p4[2] + p4[3]);
        // mnew = -inf only while every key seen by this lane was masked out
        zs[b] = mnew == -INFINITY ? 0.f : fmaf(zs[b], f, sum);
        m2[b] = mnew;
      }
    } else {
      // lane: key `col` of sub-tile kg; window rows 8*(j/4) + 4*hf + (j%4) of block b
      float p4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j) p4[j & 3] += fast_exp2(fmaf(acc[b][j], a.c, -lr[b][j]));
      red[(t & 1) * kThreads + tid] = (p4[0] + p4[1]) + (p4[2] + p4[3]);
    }
  };
  // One pipelined iteration on full tiles: the 2*KSTEPS MFMAs of tile t+1 are
  // interleaved one by one with slices of the softmax work of tile t (two
  // elements per slice), fenced so that the compiler keeps the order and the
  // matrix core and the VALU of this wave run side by side.
  auto body = [&](int t, f32x16_t(&cur)[2], f32x16_t(&nxt)[2], bf16x8_t(&kf)[KSTEPS]) {
    static_assert(2 * KSTEPS * 2 == 32 || 2 * KSTEPS * 4 == 32, "slices cover 32 elements");
    constexpr int PER = 32 / (2 * KSTEPS);  // elements of `cur` per MFMA
    wait_tiles<NLD, NBUF - 2>(min(NBUF - 2, ntiles - 2 - t));  // tile t+1 has landed
    lds_barrier();
    if (t + NBUF < ntiles) issue_tile(t + NBUF);
    if (PASS == 2 && t > 0) reduce_tile(t - 1);
    const uint32_t tb = kbuf_lds + ((t + 1) % NBUF) * TILE_BYTES;
#pragma unroll
    for (int st = 0; st < KSTEPS; ++st)
      kf[st] = lds_read_b128(tb + tile_offset<D>(kr, (D / 16) * hf + st));
    // pass 1: the tile's row maxima and the rescale factors, while LDS reads fly
    float mnew[2], fsc[2];
    if (PASS == 1) {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        float tmax = cur[b][0];
#pragma unroll
        for (int j = 1; j < 16; ++j) tmax = fmaxf(tmax, cur[b][j]);
        mnew[b] = fmaxf(m2[b], tmax * a.c);
        fsc[b] = fast_exp2(m2[b] - mnew[b]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    lds_settle(kf);
    nxt[0] = f32x16_t{};
    nxt[1] = f32x16_t{};
    float p4[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int i = 0; i < 2 * KSTEPS; ++i) {
      const int st = i >> 1, b = i & 1;
      if (PASS == 1)
        nxt[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st], qf[b][st], nxt[b], 0, 0, 0);
      else
        nxt[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[b][st], kf[st], nxt[b], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int e = i * PER; e < (i + 1) * PER; ++e) {
        const int bb = e >> 4, j = e & 15;
        const float ref = PASS == 1 ? mnew[bb] : lr[bb][j];
        p4[bb][j & 3] += fast_exp2(fmaf(cur[bb][j], a.c, -ref));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (PASS == 1) {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        // full tile: mnew is finite; fsc = 0 on the first tile (m2 = -inf)
        const float sum = (p4[b][0] + p4[b][1]) + (p4[b][2] + p4[b][3]);
        zs[b] = fmaf(zs[b], fsc[b], sum);
        m2[b] = mnew[b];
        settle(zs[b]);  // keeps this iteration's VALU work inside this iteration
      }
    } else {
      red[(t & 1) * kThreads + tid] =
          ((p4[0][0] + p4[0][1]) + (p4[0][2] + p4[0][3])) +
          ((p4[1][0] + p4[1][1]) + (p4[1][2] + p4[1][3]));
    }
  };

#pragma unroll
  for (int t = 0; t < NBUF - 1; ++t)
    if (t < ntiles) issue_tile(t);
  wait_tiles<NLD, NBUF - 2>(min(NBUF - 2, ntiles - 1));  // tile 0 has landed
  lds_barrier();
  if (NBUF - 1 < ntiles) issue_tile(NBUF - 1);
  bf16x8_t kf[KSTEPS];
  f32x16_t acc_a[2], acc_b[2];
  read_frags(0, kf);
  mfma_tile(kf, acc_a);
  int t = 0;
  for (; t + 2 < ntiles; t += 2) {  // ping-pong accumulators, no register copies
    body(t, acc_a, acc_b, kf);
    body(t + 1, acc_b, acc_a, kf);
  }
  f32x16_t(&last)[2] = (t + 1 < ntiles) ? acc_b : acc_a;
  if (t + 1 < ntiles) {
    body(t, acc_a, acc_b, kf);
    ++t;
  }
  // t = ntiles - 1: the last, possibly partial, tile
  lds_barrier();
  if (PASS == 2 && t > 0) reduce_tile(t - 1);
  finish_tile(last, t, (t + 1) * TILE <= nkeys);

  if (PASS == 2) {
    lds_barrier();
    reduce_tile(t);
    return;
  }

  // ---- pass 1 epilogue: merge lane halves, then key groups, then store
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const float mo = __shfl_xor(m2[b], 32, kWave);
    const float zo = __shfl_xor(zs[b], 32, kWave);
    const float M = fmaxf(m2[b], mo);
    float z = 0.f;
    if (M != -INFINITY) z = zs[b] * fast_exp2(m2[b] - M) + zo * fast_exp2(mo - M);
    m2[b] = M;
    zs[b] = z;
  }
  if (KG > 1) {
    float2* cm = reinterpret_cast<float2*>(red);  // [KG][RG*64]
    lds_barrier();
    if (hf == 0) {
#pragma unroll
      for (int b = 0; b < 2; ++b) cm[kg * (RG * 64) + rg * 64 + b * 32 + col] = make_float2(m2[b], zs[b]);
    }
    lds_barrier();
    if (kg == 0 && hf == 0) {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        for (int k2 = 1; k2 < KG; ++k2) {
          const float2 o = cm[k2 * (RG * 64) + rg * 64 + b * 32 + col];
          const float M = fmaxf(m2[b], o.x);
          if (M != -INFINITY) {
            zs[b] = zs[b] * fast_exp2(m2[b] - M) + o.y * fast_exp2(o.x - M);
            m2[b] = M;
          }
        }
      }
    }
  }
  if (kg == 0 && hf == 0) {
    float2* out = a.partial + ((size_t)lh * a.total_chunks + a.cu_chunks[s] + c) * a.rows_pad;
#pragma unroll
    for (int b = 0; b < 2; ++b) out[rg * 64 + b * 32 + col] = make_float2(m2[b], zs[b]);
  }
}

// Merge the per-chunk (max, sum) partials of one (sequence, head) into the
// log2-domain log-sum-exp of every window row; padding rows get +inf so
// that pass 2 gives them probability zero.
__global__ void lse_combine_kernel(SaliencyArgs a) {
  const int LH = a.L * a.Hkv;
  const int s = blockIdx.x / LH, lh = blockIdx.x - s * LH;
  const int row = threadIdx.x;
  const int c0 = a.cu_chunks[s], c1 = a.cu_chunks[s + 1];
  float M = -INFINITY, Z = 0.f;
  for (int c = c0; c < c1; ++c) {
    const float2 p = a.partial[((size_t)lh * a.total_chunks + c) * a.rows_pad + row];
    const float Mn = fmaxf(M, p.x);
    if (Mn != -INFINITY) {
      Z = Z * exp2f(M - Mn) + p.y * exp2f(p.x - Mn);
      M = Mn;
    }
  }
  a.lse2[((size_t)s * LH + lh) * a.rows_pad + row] = (row < a.R) ? M + log2f(Z) : INFINITY;
}

template <int D, int RG>
hipError_t launch_passes(const SaliencyArgs& a, hipStream_t st) {
  const int LH = a.L * a.Hkv;
  const unsigned grid = (unsigned)LH * (unsigned)a.total_chunks;
  hipLaunchKernelGGL((saliency_kernel<D, RG, 1>), dim3(grid), dim3(kThreads), 0, st, a);
  hipLaunchKernelGGL(lse_combine_kernel, dim3(a.S * LH), dim3(a.rows_pad), 0, st, a);
  hipLaunchKernelGGL((saliency_kernel<D, RG, 2>), dim3(grid), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace

int saliency_rows_pad(int R) { return R <= 64 ? 64 : (R <= 128 ? 128 : 256); }
int saliency_tile_keys(int R) { return 32 * (4 / (saliency_rows_pad(R) / 64)); }

hipError_t launch_saliency(const SaliencyArgs& a, int d, hipStream_t st) {
  hipLaunchKernelGGL(chunk_plan_kernel, dim3(1), dim3(64), 0, st, a.cu_seqlens, a.cu_chunks, a.S,
                     a.chunk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.total_chunks == 0) return e;
  const int rg = a.rows_pad / 64;
  if (d == 128) {
    if (rg == 1) return launch_passes<128, 1>(a, st);
    if (rg == 2) return launch_passes<128, 2>(a, st);
    return launch_passes<128, 4>(a, st);
  }
  if (rg == 1) return launch_passes<64, 1>(a, st);
  if (rg == 2) return launch_passes<64, 2>(a, st);
  return launch_passes<64, 4>(a, st);
}

}  // namespace stepkv
