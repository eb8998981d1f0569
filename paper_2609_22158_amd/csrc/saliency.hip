// Observation-window token saliency (Sec. 5.2, token saliency T_i):
//   A_i = sum over window rows r of softmax_i(scale * q_r . k_i)
// for every (sequence, layer, KV head), exactly, in two sweeps over K.
//
// The row softmax needs each row's log-sum-exp over all N keys before any
// column can be summed, so the kernels run
//   pass 1  per key chunk: z = K Q^T on MFMA, per-row running (max, sum exp)
//   combine per row: merge the chunk partials into log2-domain LSE
//   pass 2  per key chunk: z = Q K^T on MFMA, A_i = sum_r exp2(c z - lse_r)
// either as three launches, or in one launch (saliency_fused_kernel) whose
// column-sum chunks follow their head's row-LSE chunks about one round of
// workgroups later, so that the second read of each chunk of K is served by
// the Infinity Cache.
// The two passes swap the MFMA operands so that each reduction stays inside
// a lane: in pass 1 a lane holds 16 keys of one window row, in pass 2 16
// window rows of one key (v_mfma_f32_32x32x16_bf16 output layout).
//
// K tiles stream HBM -> LDS with global_load_lds_dwordx4 (fully coalesced,
// no VGPR round trip) into an XOR-swizzled ring of NBUF buffers; Q stays in
// VGPRs for the whole chunk. One barrier per two tiles.
#include "common.h"
#include "internal.h"

#include <math.h>

#include <type_traits>

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

// K ring per workgroup: four 8 KiB tiles at W*G = 256 rows, four 16 KiB tiles
// at 128 rows, two 32 KiB tiles at 64 rows; two workgroups per CU fit in LDS.
#ifndef STEPKV_SAL_RING_BYTES
#define STEPKV_SAL_RING_BYTES (TILE_BYTES <= 8192 ? 32768 : 65536)
#endif
// Key tiles per workgroup barrier (2: the barrier that makes tiles t+1 and t+2
// visible also frees the slots of tiles t-1 and t; 1.5-2.5% faster than one
// barrier per tile on the 32k and ragged caches).
#ifndef STEPKV_SAL_SYNC_TILES
#define STEPKV_SAL_SYNC_TILES 2
#endif
// With one barrier per two tiles: read the K fragments of tile t+2 while the
// MFMAs of tile t+1 run (each fragment register is refilled right after its
// last MFMA), so that no tile starts on an LDS round trip.
#ifndef STEPKV_SAL_FRAG_AHEAD
#define STEPKV_SAL_FRAG_AHEAD 1
#endif

// One 16-byte LDS read of the K ring at addr + OFF. Issued as assembly so
// that the compiler, which cannot tell the ring slots apart, does not put a
// vmcnt(0) (a wait for the whole prefetch ring) in front of it; completion is
// awaited explicitly with lds_wait / lds_settle.
template <int OFF>
__device__ __forceinline__ bf16x8_t lds_read_b128(uint32_t addr) {
  bf16x8_t v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF) : "memory");
  return v;
}

// Wait until at most N LDS operations of this wave are outstanding. LDS
// returns in issue order, so after issuing fragments 0..F-1 back to back,
// lds_wait<F-1-k>(frag[k]) makes fragment k (and all before it) usable.
template <int N>
__device__ __forceinline__ void lds_wait(bf16x8_t& f) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(f) : "n"(N));
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

// Key chunks of sequence s: ceil(N_s / chunk), from cu_seqlens (s may differ
// between lanes) ...
__device__ __forceinline__ int chunks_in_memory(const SaliencyArgs& a, int s) {
  return (a.cu_seqlens[s + 1] - a.cu_seqlens[s] + a.chunk - 1) / a.chunk;
}

// ... or, for a wave-uniform s, from the argument tables when the batch has them.
__device__ __forceinline__ int chunks_of(const SaliencyArgs& a, int s) {
  if (a.S <= SaliencyArgs::kArgSeqs) return a.chunk_first[s + 1] - a.chunk_first[s];
  return chunks_in_memory(a, s);
}

// The sequence s holding global chunk g (chunks of the sequences in order) and
// its first global chunk: a wave-wide prefix over 64 sequences at a time, in
// every wave (g is below the chunk total, so some sequence holds it).
__device__ __forceinline__ void locate_chunk(const SaliencyArgs& a, int g, int& s_out,
                                             int& first_out) {
  const int lane = threadIdx.x & 63;
  int base = 0;
  s_out = a.S - 1;
  first_out = 0;
  for (int s0 = 0; s0 < a.S; s0 += kWave) {
    const int sq = s0 + lane;
    const int cnt = sq < a.S ? chunks_in_memory(a, sq) : 0;
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
      first_out = base + __shfl(incl - cnt, first, kWave);
      return;
    }
    base += total;
  }
}

// Global chunk g (wave-uniform): its sequence s, the sequence's first global
// chunk, first key and length. Batches of up to kArgSeqs sequences search the
// argument tables (five scalar loads); larger ones take locate_chunk and read
// cu_seqlens.
struct ChunkLoc {
  int s, first, seq0, ns;
};

__device__ __forceinline__ ChunkLoc find_chunk(const SaliencyArgs& a, int g) {
  ChunkLoc r;
  if (a.S <= SaliencyArgs::kArgSeqs) {
    // the last s with chunk_first[s] <= g (a sequence without keys has no
    // chunk, so the search passes over it)
    int lo = 0;
#pragma unroll
    for (int step = SaliencyArgs::kArgSeqs / 2; step > 0; step >>= 1)
      if (a.chunk_first[lo + step] <= g) lo += step;
    r.s = lo;
    r.first = a.chunk_first[lo];
    r.seq0 = a.seq_first[lo];
    r.ns = a.seq_first[lo + 1] - r.seq0;
  } else {
    locate_chunk(a, g, r.s, r.first);
    r.s = uniform(r.s);
    r.first = uniform(r.first);
    // read into scalar registers: a value either branch may give stays scalar
    r.seq0 = uniform(a.cu_seqlens[r.s]);
    r.ns = uniform(a.cu_seqlens[r.s + 1]) - r.seq0;
  }
  return r;
}

// The first global chunk of sequence s: the chunks of the sequences before it.
__device__ __forceinline__ int first_chunk(const SaliencyArgs& a, int s) {
  if (a.S <= SaliencyArgs::kArgSeqs) return a.chunk_first[s];
  const int lane = threadIdx.x & 63;
  int acc = 0;
  for (int s0 = 0; s0 < s; s0 += kWave) {
    int cnt = s0 + lane < s ? chunks_in_memory(a, s0 + lane) : 0;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off, kWave);
    acc += cnt;
  }
  return acc;
}

// Calls f(std::integral_constant<int, I>{}) for I = B .. E-1, unrolled.
template <int B, int E, typename F>
__host__ __device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// D: head dim. RG: row groups of 64 window rows (1, 2 or 4); the 4 / RG
// waves per row group split each key tile into 32-key sub-tiles. CAUSAL:
// window slot w sees keys up to N_s - W + w only (the mask code exists only
// in these instantiations).
//
// The tile loop is unrolled by the ring depth so that every ring slot is a
// compile-time LDS offset: fragment reads use per-lane addresses computed
// once plus an immediate, and full tiles load from a scalar base plus
// per-lane constant offsets.
// Device-coherent accesses (relaxed atomics at agent scope: they bypass the
// per-XCD L2) for the few values that one workgroup of the one-launch sweeps
// hands to another: the chunk partials, the row LSEs and the counters. A
// writer waits for its stores (vmcnt 0) before it moves a counter, and a
// reader issues its loads after it has seen the counter, so no L2 write-back
// or invalidation is needed around them.
__device__ __forceinline__ void store_coherent(float2* p, float2 v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), __builtin_bit_cast(uint64_t, v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_coherent(float* p, float v) {
  __hip_atomic_store(reinterpret_cast<uint32_t*>(p), __builtin_bit_cast(uint32_t, v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 load_coherent(const float2* p) {
  return __builtin_bit_cast(float2, __hip_atomic_load(reinterpret_cast<const uint64_t*>(p),
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ float load_coherent(const float* p) {
  return __builtin_bit_cast(float, __hip_atomic_load(reinterpret_cast<const uint32_t*>(p),
                                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
// This wave's stores have completed.
__device__ __forceinline__ void stores_done() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Compile-time shape of the sweeps for head dim D and RG row groups: the K
// ring (NBUF tiles of TILE keys) and the LDS buffers of the column partials.
template <int D, int RG>
struct SweepShape {
  static constexpr int KG = 4 / RG;
  static constexpr int TILE = 32 * KG;               // keys per workgroup iteration
  static constexpr int KSTEPS = D / 16;              // MFMA k-steps
  static constexpr int TILE_BYTES = TILE * 2 * D;
  // ring slots: an even count, 2 to 8, within STEPKV_SAL_RING_BYTES
  static constexpr int NBUF_FIT = STEPKV_SAL_RING_BYTES / TILE_BYTES;
  static constexpr int NBUF = NBUF_FIT >= 8 ? 8 : (NBUF_FIT >= 2 ? NBUF_FIT & ~1 : 2);
  static constexpr int NLD = TILE_BYTES / (kThreads * 16);  // 16-byte loads per thread per tile
  // tiles per workgroup barrier: 1, or 2 when the ring holds at least 4 tiles
  static constexpr int SYNC = (STEPKV_SAL_SYNC_TILES == 2 && NBUF >= 4) ? 2 : 1;
  static constexpr int NRED = 2 * SYNC;  // column-partial buffers of the second sweep
  static constexpr int RING_BYTES = NBUF * TILE_BYTES;
  static constexpr int RED_FLOATS = NRED * kThreads;
};

// One sweep over one key chunk: global chunk g (the chunks of all sequences in
// order) of head lh, with the workgroup's K ring and partial buffers in LDS.
// PASS 1 writes the chunk's per-row (max, sum) partials, PASS 2 the chunk's
// column sums (from the row LSEs in a.lse2).
// FUSED (both sweeps in one launch): the first sweep's K loads keep their
// lines in the caches, where the second sweep reads the chunk again, and the
// partials and row LSEs that pass between workgroups use device-coherent
// accesses. Otherwise every K load is non-temporal, which leaves the caches to
// the saliency the second sweep writes and the priority reads next.
template <int D, int RG, int PASS, bool CAUSAL, bool FUSED, typename BeforeLse>
__device__ __forceinline__ void sweep(const SaliencyArgs& a, int lh, const int rem_blk,
                                      const ChunkLoc& loc, uint8_t* __restrict__ kbuf,
                                      float* __restrict__ red, BeforeLse&& before_lse) {
  using Sh = SweepShape<D, RG>;
  constexpr int KG = Sh::KG;
  constexpr int TILE = Sh::TILE;
  constexpr int KSTEPS = Sh::KSTEPS;
  constexpr int TILE_BYTES = Sh::TILE_BYTES;
  constexpr int NBUF = Sh::NBUF;
  constexpr int NLD = Sh::NLD;
  static_assert(NLD >= 1, "tile too small");
  static_assert((NBUF - 1) * TILE_BYTES < 65536, "ring offset must fit the ds_read offset field");
  constexpr int SYNC = Sh::SYNC;
  // fragments one tile ahead (needs the two-tile barrier: a barrier at even
  // tile t makes tiles t+2 and t+3 visible, read in bodies t and t+1)
  constexpr bool AHEAD = SYNC == 2 && (STEPKV_SAL_FRAG_AHEAD == 2 ||
                                        (STEPKV_SAL_FRAG_AHEAD == 1 && PASS == 1 && RG == 4 && !CAUSAL));
  constexpr int NRED = Sh::NRED;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int rg = wave % RG, kg = wave / RG;
  const int col = lane & 31, hf = lane >> 5;

  // ---- work item: (head lh, sequence s, chunk c)
  const int LH = a.L * a.Hkv;
  const int s = loc.s;
  const int c = uniform(rem_blk - loc.first);
  const int l = lh / a.Hkv, h = lh - l * a.Hkv;
  const int seq0 = loc.seq0;
  const int ns = loc.ns;
  const int key0 = c * a.chunk;
  const int nkeys = min(a.chunk, ns - key0);
  const int ntiles = (nkeys + TILE - 1) / TILE;
  const uint16_t* __restrict__ kseq = a.k + ((size_t)lh * a.ntot + seq0) * D;

  // ---- K ring: this lane's 16-byte pieces of a tile (HBM side) ...
  const char* __restrict__ kbytes = reinterpret_cast<const char*>(kseq);
  uint32_t ld_off[NLD];  // byte offset from the tile's first key row
  int ld_row[NLD];       // key row inside the tile
#pragma unroll
  for (int j = 0; j < NLD; ++j) {
    const int o = 16 * (tid + kThreads * j);
    const int r = o / (2 * D);
    const int p = ((o % (2 * D)) / 16) ^ swizzle<D>(r);
    ld_row[j] = r;
    ld_off[j] = r * (2 * D) + 16 * p;
  }
  // ... and the LDS side: fragment st of this lane's key row
  const uint32_t kbuf_lds = static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t*)kbuf));
  const int kr = kg * 32 + col;
  uint32_t fa[KSTEPS];
#pragma unroll
  for (int st = 0; st < KSTEPS; ++st) fa[st] = kbuf_lds + tile_offset<D>(kr, (D / 16) * hf + st);

  auto issue_tile = [&](int t, auto slot_c) __attribute__((always_inline)) {
    constexpr int slot = decltype(slot_c)::value;
    const int kt = key0 + t * TILE;  // first key of the tile
    uint8_t* base = kbuf + slot * TILE_BYTES;
    if (kt + TILE <= ns) {
      const char* tb = kbytes + (size_t)kt * (2 * D);
#pragma unroll
      for (int j = 0; j < NLD; ++j)
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(tb + ld_off[j]),
                                         (__attribute__((address_space(3))) void*)(
                                             base + 16 * (kThreads * j + 64 * wave)),
                                         16, 0, FUSED && PASS == 1 ? 0 : 2);
    } else {  // tail rows re-read the last valid key
#pragma unroll
      for (int j = 0; j < NLD; ++j) {
        const int key = min(kt + ld_row[j], ns - 1);
        const char* src = kbytes + (size_t)key * (2 * D) + (ld_off[j] - ld_row[j] * (2 * D));
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(src),
                                         (__attribute__((address_space(3))) void*)(
                                             base + 16 * (kThreads * j + 64 * wave)),
                                         16, 0, FUSED && PASS == 1 ? 0 : 2);
      }
    }
  };
  auto read_frags = [&](auto slot_c, bf16x8_t(&kf)[KSTEPS]) __attribute__((always_inline)) {
    constexpr int slot = decltype(slot_c)::value;
#pragma unroll
    for (int st = 0; st < KSTEPS; ++st) kf[st] = lds_read_b128<slot * TILE_BYTES>(fa[st]);
  };

  // The first K tiles go out before the window rows of Q, so that a chunk
  // starts after one memory round trip, not two. With fragments one tile ahead
  // every slot fills now (tiles 0 and 1 must land), otherwise all but the last
  // (it fills at tile 0's barrier, or below with one barrier per tile).
  static_for<0, AHEAD ? NBUF : NBUF - 1>([&](auto ic) __attribute__((always_inline)) {
    if (decltype(ic)::value < ntiles) issue_tile(decltype(ic)::value, ic);
  });

  // ---- window rows of this wave: two 32-row blocks of the launch's row group
  // (rows row0 + local row), k-slices (D/2)*hf + 8*st
  bf16x8_t qf[2][KSTEPS];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int row = rg * 64 + b * 32 + col;
    if (row < a.R) {
      const int w = (a.row0 + row) / a.G, g = (a.row0 + row) - w * a.G;
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

  // the caller's step before the row LSEs are read (the wait of a column-sum
  // chunk for its head's row LSEs in the one-launch sweeps)
  before_lse();

  // pass 1 state: per lane and row block, a log2-domain reference m2 and the
  // sum of exp2(c z - m2) over the keys seen so far (the pair stands for
  // 2^m2 * zs). Full tiles keep m2 and only move it up to the tile's maximum,
  // rescaling the sum, when the sum would exceed 2^64.
  float m2[2] = {-INFINITY, -INFINITY};
  float zs[2] = {0.f, 0.f};
  // pass 2 state: log2-domain LSE of the 16 rows this lane holds per block
  float lr[2][16];
  if (PASS == 2) {
    const float* lp = a.lse2 + ((size_t)s * LH + lh) * a.rows_pad + rg * 64;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float* e = lp + b * 32 + 8 * (j >> 2) + 4 * hf + (j & 3);
        lr[b][j] = FUSED ? load_coherent(e) : *e;
      }
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

  auto reduce_tile = [&](int t) __attribute__((always_inline)) {  // pass 2: sum the per-wave column partials of tile t
    if (tid < TILE) {
      const int kg2 = tid >> 5, col2 = tid & 31;
      const float* rp = red + (t % NRED) * kThreads;
      float sum = 0.f;
#pragma unroll
      for (int r2 = 0; r2 < RG; ++r2) {
        const int w2 = kg2 * RG + r2;
        sum += rp[w2 * 64 + col2];
        sum += rp[w2 * 64 + 32 + col2];
      }
      const int key = t * TILE + tid;
      if (key < nkeys) {
        float* o = a.sal + (size_t)lh * a.ntot + seq0 + key0 + key;
        *o = a.accumulate ? *o + sum : sum;
      }
    }
  };

  // Causal tail: key i of the sequence is visible to window slot w only when
  // i <= N_s - W + w. Only tiles reaching past N_s - W have hidden entries;
  // their logits become -inf, which every later step maps to probability 0.
  const int hidden_from = ns - a.W + 1;  // first key hidden from some window slot
  auto tile_has_hidden = [&](int t) __attribute__((always_inline)) {
    return CAUSAL && key0 + (t + 1) * TILE > hidden_from;
  };
  auto mask_hidden = [&](f32x16_t(&acc)[2], int t) __attribute__((always_inline)) {
    // key kin of the tile is visible to window row `row` (row0 + the local row)
    // iff kin <= lim + row / G
    const int lim = ns - a.W - key0 - t * TILE;
    if (PASS == 1) {  // lane: one row per block; keys kg*32 + 4*hf + 8*(j/4) + (j%4)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int thr = lim + (a.row0 + rg * 64 + b * 32 + col) / a.G - kg * 32 - 4 * hf;
#pragma unroll
        for (int j = 0; j < 16; ++j)
          if (8 * (j >> 2) + (j & 3) > thr) acc[b][j] = -INFINITY;
      }
    } else {  // lane: key kg*32 + col; rows rg*64 + 4*hf + 32*b + 8*(j/4) + (j%4)
      // row / G >= kin - lim  <=>  row >= G * (kin - lim)
      const int thr = a.G * (kg * 32 + col - lim) - a.row0 - rg * 64 - 4 * hf;
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j)
          if (b * 32 + 8 * (j >> 2) + (j & 3) < thr) acc[b][j] = -INFINITY;
    }
  };
  auto mfma_tile = [&](const bf16x8_t(&kf)[KSTEPS], f32x16_t(&acc)[2]) __attribute__((always_inline)) {
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
  // Softmax work on the last tile t, which may be partial (exact maxima).
  auto finish_tile = [&](const f32x16_t(&acc)[2], int t, bool full) __attribute__((always_inline)) {
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
      red[(t % NRED) * kThreads + tid] = (p4[0] + p4[1]) + (p4[2] + p4[3]);
    }
  };

  // One pipelined iteration on full tiles, ring slot i = t % NBUF: the
  // 2*KSTEPS MFMAs of tile t+1 are interleaved one by one with slices of the
  // softmax work of tile t (two elements per slice at D = 128), fenced so
  // that the matrix core and the VALU of this wave run side by side. Each
  // k-step waits only for its own K fragment. In pass 2 one wave per tile
  // (rotating) sums the column partials of tile t-1: its LDS reads are issued
  // first and consumed last.
  // NB: row blocks of this wave that hold window rows (2, or 1 when the second
  // is padding past R: its MFMAs and softmax work are skipped; the result is
  // the same, as padding rows contribute exact zeros)
  bf16x8_t kf[KSTEPS];  // K fragments of the tile whose MFMAs run next
  auto body = [&](auto ic, int t, f32x16_t(&cur)[2], f32x16_t(&nxt)[2], auto nb_c) __attribute__((always_inline)) {
    constexpr int i = decltype(ic)::value;
    constexpr int NB = decltype(nb_c)::value;
    constexpr int PER = 32 / (2 * KSTEPS);  // elements of `cur` per MFMA
    static_assert(PER * 2 * KSTEPS == 32, "slices cover 32 elements");
    if constexpr (SYNC == 1) {
      // tile t+1 has landed; the tiles issued after it may still be in flight
      wait_tiles<NLD, NBUF - 2>(min(NBUF - 2, ntiles - 2 - t));
      lds_barrier();
      if (t + NBUF < ntiles) issue_tile(t + NBUF, ic);  // into the slot tile t has left
    } else if constexpr (i % 2 == 0 && AHEAD) {
      // one barrier per two tiles, fragments one tile ahead: tiles t+2 and t+3
      // have landed (those that exist); every wave holds tile t+1's fragments
      // (read in the body before), so the slots of tiles t and t+1 take new tiles
      wait_tiles<NLD, NBUF - 4>(max(0, min(NBUF - 4, ntiles - 4 - t)));
      lds_barrier();
      if (t + NBUF < ntiles) issue_tile(t + NBUF, ic);
      if (t + NBUF + 1 < ntiles)
        issue_tile(t + NBUF + 1, std::integral_constant<int, (i + 1) % NBUF>{});
    } else if constexpr (i % 2 == 0) {
      // one barrier per two tiles: tiles t+1 and t+2 have landed (t+2 when it
      // exists); after the barrier every wave is done with tiles t-1 and t, so
      // both their slots take new tiles
      wait_tiles<NLD, NBUF - 4>(max(0, min(NBUF - 4, ntiles - 3 - t)));
      lds_barrier();
      if (t + NBUF - 1 < ntiles)
        issue_tile(t + NBUF - 1, std::integral_constant<int, (i + NBUF - 1) % NBUF>{});
      if (t + NBUF < ntiles) issue_tile(t + NBUF, ic);
    }
    // the column partials this wave sums: of tile t-1 (one barrier per tile), or
    // of tile t-2 or t-1 after a barrier (one per two tiles); one wave per tile,
    // rotating
    constexpr bool RED_HERE = SYNC == 1 || i % 2 == 0;
    int rt = -1;       // tile whose partials this wave sums
    int rtid = TILE;   // its key within that tile (>= TILE: none)
    if constexpr (RED_HERE) {
      // per two tiles: rotated thread index ra < TILE sums tile t-2 (key ra);
      // the threads with ra in [256 - SHIFT, 256 - SHIFT + TILE) sum tile t-1
      // (key rb = ra + SHIFT - 256): another wave for tiles of up to 64 keys,
      // the other half of the threads for 128-key tiles
      constexpr int SHIFT = TILE <= 64 ? 64 : 128;
      static_assert(SYNC == 1 || TILE <= 128, "two tiles per barrier need 2 * TILE <= 256 threads");
      const int ra = (tid + 64 * i) & (kThreads - 1);
      const int rb = (ra + SHIFT) & (kThreads - 1);
      if (SYNC == 1) {
        rt = t - 1;
        rtid = ra;
      } else if (ra < TILE) {
        rt = t - 2;
        rtid = ra;
      } else {
        rt = t - 1;
        rtid = rb;
      }
    }
    const bool reducer = PASS == 2 && RED_HERE && rt >= 0 && rtid < TILE;
    float part[2 * RG];
    if (reducer) {
      const int kg2 = rtid >> 5, col2 = rtid & 31;
      const float* rp = red + (rt % NRED) * kThreads;
#pragma unroll
      for (int r2 = 0; r2 < RG; ++r2) {
        part[2 * r2] = rp[(kg2 * RG + r2) * 64 + col2];
        part[2 * r2 + 1] = rp[(kg2 * RG + r2) * 64 + 32 + col2];
      }
    }
    if constexpr (!AHEAD) read_frags(std::integral_constant<int, (i + 1) % NBUF>{}, kf);
    if (tile_has_hidden(t)) mask_hidden(cur, t);
    __builtin_amdgcn_sched_barrier(0);
    nxt[0] = f32x16_t{};
    nxt[1] = f32x16_t{};
    float p4[2][4];
    // pass-1 reference of this tile: m2, or 0 while m2 is -inf (then every key
    // of this lane is hidden, in this tile and all later ones: the causal
    // limit is a prefix of the keys and tile 0 set m2 from its visible keys)
    float ref1[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) ref1[b] = m2[b] == -INFINITY ? 0.f : m2[b];
    // The softmax work of slice s runs in three stages one MFMA apart: the
    // scaled logit (in place in `cur`) after MFMA s, its exp2 after MFMA s+1
    // and the sum after MFMA s+2, so that no VALU instruction waits on one
    // issued just before it.
    float ex[2][PER];
    auto stage_logit = [&](auto sc) __attribute__((always_inline)) {
      constexpr int sl = decltype(sc)::value;
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int e = sl * PER + q, bb = e >> 4, j = e & 15;
        cur[bb][j] = fmaf(cur[bb][j], a.c, -(PASS == 1 ? ref1[bb] : lr[bb][j]));
      }
    };
    auto stage_exp = [&](auto sc) __attribute__((always_inline)) {
      constexpr int sl = decltype(sc)::value;
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int e = sl * PER + q, bb = e >> 4, j = e & 15;
        ex[sl & 1][q] = fast_exp2(cur[bb][j]);
      }
    };
    auto stage_sum = [&](auto sc) __attribute__((always_inline)) {
      constexpr int sl = decltype(sc)::value;
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int e = sl * PER + q, bb = e >> 4, j = e & 15;
        p4[bb][j & 3] = j < 4 ? ex[sl & 1][q] : p4[bb][j & 3] + ex[sl & 1][q];  // first touch needs no add
      }
    };
    constexpr int NSL = NB * KSTEPS;  // slices, one per MFMA
    static_for<0, NSL>([&](auto i2c) __attribute__((always_inline)) {
      constexpr int i2 = decltype(i2c)::value;
      constexpr int st = NB == 2 ? i2 >> 1 : i2, b = NB == 2 ? i2 & 1 : 0;
      if constexpr (b == 0 && !AHEAD) lds_wait<KSTEPS - 1 - st>(kf[st]);
      if (PASS == 1)
        nxt[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st], qf[b][st], nxt[b], 0, 0, 0);
      else
        nxt[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[b][st], kf[st], nxt[b], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (i2 >= 2) stage_sum(std::integral_constant<int, i2 - 2>{});
      if constexpr (i2 >= 1) stage_exp(std::integral_constant<int, i2 - 1>{});
      stage_logit(i2c);
      // the register of fragment st is free after its last MFMA: refill it with
      // tile t+2's fragment (a stale slot when t+2 is past the chunk; never used)
      if constexpr (AHEAD && b == NB - 1)
        kf[st] = lds_read_b128<((i + 2) % NBUF) * TILE_BYTES>(fa[st]);
      __builtin_amdgcn_sched_barrier(0);
    });
    stage_exp(std::integral_constant<int, NSL - 1>{});
    stage_sum(std::integral_constant<int, NSL - 2>{});
    stage_sum(std::integral_constant<int, NSL - 1>{});
    // tile t+2's fragments are complete before any branch: a value still in
    // flight must not reach code where the compiler may copy its register
    if constexpr (AHEAD) lds_settle(kf);
    // every partial sum is formed here, inside the MFMA sequence: without this
    // the compiler sinks block 1's work past block 0's branch below
    if constexpr (NB == 1) {
#pragma unroll
      for (int k = 0; k < 4; ++k) p4[1][k] = 0.f;  // the padding block adds exact zeros
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int k = 0; k < 4; ++k) settle(p4[b][k]);
    if (PASS == 1) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const float sum = (p4[b][0] + p4[b][1]) + (p4[b][2] + p4[b][3]);
        const float nz = zs[b] + sum;
        // keeps every later merge of (m2, zs) pairs finite; otherwise (too large
        // or not finite under the current reference) the reference moves to
        // this tile's max. Wave-uniform branch, lane selects inside: the
        // common path leaves the execution mask alone.
        const bool big = !(nz <= 0x1p64f);
        float znew = nz;
        if (__builtin_amdgcn_ballot_w64(big) != 0) {
          float tmax = cur[b][0];  // cur holds c*z - ref1 now
#pragma unroll
          for (int j = 1; j < 16; ++j) tmax = fmaxf(tmax, cur[b][j]);
          const float mnew = fmaxf(m2[b], ref1[b] + tmax);
          const float sh = mnew - ref1[b];
          float q4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int j = 0; j < 16; ++j) q4[j & 3] += fast_exp2(cur[b][j] - sh);
          const float moved = fmaf(zs[b], fast_exp2(m2[b] - mnew), (q4[0] + q4[1]) + (q4[2] + q4[3]));
          const bool mv = big && mnew != -INFINITY;  // -inf: every key this lane has seen is hidden
          znew = mv ? moved : (big ? zs[b] : nz);
          m2[b] = mv ? mnew : m2[b];
        }
        zs[b] = znew;
        settle(zs[b]);  // keeps this iteration's VALU work inside this iteration
      }
    } else {
      red[(t % NRED) * kThreads + tid] =
          ((p4[0][0] + p4[0][1]) + (p4[0][2] + p4[0][3])) +
          ((p4[1][0] + p4[1][1]) + (p4[1][2] + p4[1][3]));
      if (reducer) {  // tile rt < t is full: only the last tile can be partial
#pragma unroll
        for (int k2 = 0; k2 < 2 * RG; ++k2) settle(part[k2]);  // consume the reads here, late
        float sum = part[0];
#pragma unroll
        for (int k2 = 1; k2 < 2 * RG; ++k2) sum += part[k2];
        float* o = a.sal + (size_t)lh * a.ntot + seq0 + key0 + rt * TILE + rtid;
        *o = a.accumulate ? *o + sum : sum;
      }
    }
  };

  if constexpr (AHEAD)
    wait_tiles<NLD, NBUF - 2>(max(0, min(NBUF - 2, ntiles - 2)));  // tiles 0 and 1 have landed
  else
    wait_tiles<NLD, NBUF - 2>(min(NBUF - 2, ntiles - 1));  // tile 0 has landed
  lds_barrier();
  if (SYNC == 1 && NBUF - 1 < ntiles) issue_tile(NBUF - 1, std::integral_constant<int, NBUF - 1>{});
  f32x16_t acc_a[2], acc_b[2];
  read_frags(std::integral_constant<int, 0>{}, kf);
  lds_settle(kf);
  mfma_tile(kf, acc_a);
  // tile 1's fragments for the first body (a stale slot when there is no tile 1)
  if constexpr (AHEAD) {
    read_frags(std::integral_constant<int, 1>{}, kf);
    lds_settle(kf);
  }
  if (PASS == 1 && ntiles > 1) {  // tile 0 is full: its maxima are the first references
    if (tile_has_hidden(0)) mask_hidden(acc_a, 0);
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      float tmax = acc_a[b][0];
#pragma unroll
      for (int j = 1; j < 16; ++j) tmax = fmaxf(tmax, acc_a[b][j]);
      m2[b] = tmax * a.c;
    }
  }
  int t = 0, rest = 0;
  auto tiles = [&](auto nb_c) __attribute__((always_inline)) {
    for (; t + NBUF < ntiles; t += NBUF) {  // ping-pong accumulators, no register copies
      static_for<0, NBUF>([&](auto ic) __attribute__((always_inline)) {
        if constexpr (decltype(ic)::value % 2 == 0)
          body(ic, t + decltype(ic)::value, acc_a, acc_b, nb_c);
        else
          body(ic, t + decltype(ic)::value, acc_b, acc_a, nb_c);
      });
    }
    rest = ntiles - 1 - t;  // 0 .. NBUF-1 full tiles before the last one
    static_for<0, NBUF - 1>([&](auto ic) __attribute__((always_inline)) {
      if (decltype(ic)::value < rest) {
        if constexpr (decltype(ic)::value % 2 == 0)
          body(ic, t + decltype(ic)::value, acc_a, acc_b, nb_c);
        else
          body(ic, t + decltype(ic)::value, acc_b, acc_a, nb_c);
      }
    });
  };
  // wave-uniform: whether this wave's second row block holds any window row
  if (rg * 64 + 32 < a.R) tiles(std::integral_constant<int, 2>{});
  else tiles(std::integral_constant<int, 1>{});
  t += rest;
  f32x16_t(&last)[2] = (rest & 1) ? acc_b : acc_a;
  // t = ntiles - 1: the last, possibly partial, tile
  lds_barrier();
  if (PASS == 2) {  // the full tiles whose partials no barrier has covered yet
    if (SYNC == 1) {
      if (t > 0) reduce_tile(t - 1);
    } else {
      // partials of tiles up to e - 1 were summed at the last barrier e (even, <= t - 1)
      const int e = t >= 1 ? ((t - 1) & ~1) : 0;
      for (int x = e; x < t; ++x) reduce_tile(x);
    }
  }
  f32x16_t fin[2] = {last[0], last[1]};  // a copy: writing through `last` would demote both
  if (tile_has_hidden(t)) mask_hidden(fin, t);
  finish_tile(fin, t, (t + 1) * TILE <= nkeys);

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
    float2* out = a.partial + ((size_t)lh * a.total_chunks + rem_blk) * a.rows_pad;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      float2* e = out + rg * 64 + b * 32 + col;
      if (FUSED) store_coherent(e, make_float2(m2[b], zs[b]));
      else *e = make_float2(m2[b], zs[b]);
    }
  }
}

// One launch per sweep: block b takes chunk b % total_chunks of head
// b / total_chunks (the column-sum sweep walks the heads in reverse, so that
// it starts on the heads the row-LSE sweep read last).
template <int D, int RG, int PASS, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 2) void saliency_kernel(SaliencyArgs a) {
  using Sh = SweepShape<D, RG>;
  __shared__ __attribute__((aligned(16))) uint8_t kbuf[Sh::RING_BYTES];
  __shared__ float red[Sh::RED_FLOATS];
  const int LH = a.L * a.Hkv;
  int lh = blockIdx.x / a.total_chunks;
  const int g = blockIdx.x - lh * a.total_chunks;
  if (PASS == 2) lh = LH - 1 - lh;
  sweep<D, RG, PASS, CAUSAL, false>(a, lh, g, find_chunk(a, g), kbuf, red, [] {});
}

// The log2-domain row LSE from a row's merged (max, sum): +inf for padding
// rows and rows that see no key (probability zero in the second sweep); the
// natural-log value of every real row is exported when lse_out is set (-inf
// for a row that sees no key).
template <bool COHERENT>
__device__ __forceinline__ void store_row_lse(const SaliencyArgs& a, int s, int lh, int row,
                                              float M, float Z) {
  const int LH = a.L * a.Hkv;
  const bool seen = row < a.R && Z > 0.f;
  const float l2 = seen ? M + log2f(Z) : INFINITY;
  float* e = a.lse2 + ((size_t)s * LH + lh) * a.rows_pad + row;
  if (COHERENT) store_coherent(e, l2);
  else *e = l2;
  if (a.lse_out && row < a.R) {
    const int l = lh / a.Hkv, h = lh - l * a.Hkv;
    const int w = (a.row0 + row) / a.G, g = (a.row0 + row) - w * a.G;
    a.lse_out[(((size_t)l * a.S + s) * a.W + w) * a.Hq + h * a.G + g] =
        seen ? l2 * 0.693147180559945309f : -INFINITY;
  }
}

// ---- both sweeps in one launch, K read once from HBM
//
// Work items are the chunks of both sweeps. The row-LSE items of every
// (sequence, head) come first in item order and its column-sum items follow
// about one round of resident workgroups later, so that the K they read
// again is still in the Infinity Cache: item t of the launch is
//   t < lag:               row-LSE item t
//   lag <= t < 2M - lag:   row-LSE item lag + (t - lag) / 2 (t - lag even),
//                          column-sum item (t - lag - 1) / 2 (t - lag odd)
//   t >= 2M - lag:         column-sum item t - M
// with M items per sweep, in the order head-major, chunks of the sequences in
// order. The column-sum item k follows the row-LSE items of its (sequence,
// head) in this order when lag is at least the most chunks of a sequence.
//
// Each (sequence, head) has a counter: every row-LSE item adds one after its
// partials have reached device-coherent memory; the one that completes the
// count merges the partials into the row LSEs and adds one more. A column-sum item waits
// for count = chunks + 1. Blocks start in index order, so every row-LSE item
// a column-sum item waits for has started and finishes without waiting; the
// wait is still bounded (kFusedSpins polls), and one that runs out sets
// STEPKV_FLAG_SYNC in the status word and goes on.
constexpr int kFusedSpins = 1 << 17;

__device__ __forceinline__ void fused_item(int t, int M, int lag, int& pass, int& k) {
  if (t < lag) {
    pass = 1;
    k = t;
  } else if (t < 2 * M - lag) {
    const int j = t - lag;
    pass = (j & 1) ? 2 : 1;
    k = (j & 1) ? (j >> 1) : lag + (j >> 1);
  } else {
    pass = 2;
    k = t - M;
  }
}

// Row LSEs of (s, lh) from the partials of its nch chunks from global chunk
// c0 on: one thread per row, the chunks in order, eight loads in flight.
__device__ __forceinline__ void merge_unit(const SaliencyArgs& a, int s, int lh, int c0,
                                           int nch) {
  const int row = threadIdx.x;
  if (row >= a.rows_pad) return;
  const float2* __restrict__ pp =
      a.partial + ((size_t)lh * a.total_chunks + c0) * a.rows_pad + row;
  float M = -INFINITY, Z = 0.f;
  for (int c = 0; c < nch; c += 8) {
    float2 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      v[u] = c + u < nch ? load_coherent(pp + (size_t)(c + u) * a.rows_pad)
                         : make_float2(-INFINITY, 0.f);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float Mn = fmaxf(M, v[u].x);
      if (Mn != -INFINITY) {
        Z = Z * exp2f(M - Mn) + v[u].y * exp2f(v[u].x - Mn);
        M = Mn;
      }
    }
  }
  store_row_lse<true>(a, s, lh, row, M, Z);
}

template <int D, int RG, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 2) void saliency_fused_kernel(SaliencyArgs a) {
  using Sh = SweepShape<D, RG>;
  __shared__ __attribute__((aligned(16))) uint8_t kbuf[Sh::RING_BYTES];
  __shared__ float red[Sh::RED_FLOATS];
  __shared__ int last;
  const int LH = a.L * a.Hkv;
  const int M = LH * a.total_chunks;
  int pass, k;
  fused_item((int)blockIdx.x, M, a.lag, pass, k);
  pass = uniform(pass);
  k = uniform(k);
  const int lh = k / a.total_chunks, g = k - lh * a.total_chunks;
  const ChunkLoc loc = find_chunk(a, g);
  const int s = loc.s, c0 = loc.first;
  const int nch = chunks_of(a, s);
  int* cnt = a.unit_cnt + (size_t)s * LH + lh;
  if (pass == 1) {
    sweep<D, RG, 1, CAUSAL, true>(a, lh, g, loc, kbuf, red, [] {});
    // this wave's partials have reached device-coherent memory before the count moves
    stores_done();
    __syncthreads();
    if (threadIdx.x == 0)
      last = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nch - 1;
    __syncthreads();
    if (!last) return;
    merge_unit(a, s, lh, c0, nch);
    stores_done();
    __syncthreads();
    if (threadIdx.x == 0) __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  } else {
    // the chunk's first K tiles and Q are on their way while this waits
    sweep<D, RG, 2, CAUSAL, true>(a, lh, g, loc, kbuf, red, [&] {
      if (threadIdx.x == 0) {
        int spins = 0;
        while (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < nch + 1) {
          __builtin_amdgcn_s_sleep(2);
          if (++spins == kFusedSpins) {
            if (a.status) atomicOr(a.status, kFlagSync);
            break;
          }
        }
      }
      __syncthreads();
    });
  }
}

// Merge the per-chunk (max, sum) partials of one (sequence, head) into the
// log2-domain log-sum-exp of every window row (store_row_lse).
// 1024 threads per (sequence, head): each row's chunks are split over
// 1024 / rows_pad groups, each taking one online pass over its chunks with
// eight loads in flight, and the groups are merged in LDS.
constexpr int kCombineThreads = 1024;

__global__ __launch_bounds__(kCombineThreads) void lse_combine_kernel(SaliencyArgs a) {
  __shared__ float2 part[kCombineThreads];
  const int LH = a.L * a.Hkv;
  const int s = blockIdx.x / LH, lh = blockIdx.x - s * LH;
  const int row = threadIdx.x % a.rows_pad, grp = threadIdx.x / a.rows_pad;
  const int ngrp = kCombineThreads / a.rows_pad;
  const int c0 = first_chunk(a, s), c1 = c0 + chunks_of(a, s);
  const float2* __restrict__ pp = a.partial + (size_t)lh * a.total_chunks * a.rows_pad + row;
  // one online pass over this thread's chunks, eight loads in flight at a time;
  // a chunk whose keys this row never saw is (-inf, 0) and adds nothing
  float M = -INFINITY, Z = 0.f;
  for (int c = c0 + grp; c < c1; c += 8 * ngrp) {
    float2 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int cc = c + u * ngrp;
      v[u] = cc < c1 ? pp[(size_t)cc * a.rows_pad] : make_float2(-INFINITY, 0.f);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float Mn = fmaxf(M, v[u].x);
      if (Mn != -INFINITY) {
        Z = Z * exp2f(M - Mn) + v[u].y * exp2f(v[u].x - Mn);
        M = Mn;
      }
    }
  }
  part[threadIdx.x] = make_float2(M, Z);
  __syncthreads();
  if (grp != 0) return;
  for (int g = 1; g < ngrp; ++g) {
    const float2 o = part[g * a.rows_pad + row];
    const float Mn = fmaxf(M, o.x);
    if (Mn != -INFINITY) {
      Z = Z * exp2f(M - Mn) + o.y * exp2f(o.x - Mn);
      M = Mn;
    }
  }
  store_row_lse<false>(a, s, lh, row, M, Z);
}

// The caller's natural-log row LSE (lse_in [L][S][W][Hq]) in the layout and
// log2 domain of the second sweep; -inf (a row that sees no key) and padding
// rows become +inf.
__global__ void lse_import_kernel(SaliencyArgs a) {
  const int LH = a.L * a.Hkv;
  const int s = blockIdx.x / LH, lh = blockIdx.x - s * LH;
  const int row = threadIdx.x;
  float l2 = INFINITY;
  if (row < a.R) {
    const int l = lh / a.Hkv, h = lh - l * a.Hkv;
    const int w = (a.row0 + row) / a.G, g = (a.row0 + row) - w * a.G;
    const float x = a.lse_in[(((size_t)l * a.S + s) * a.W + w) * a.Hq + h * a.G + g];
    if (x != -INFINITY) l2 = x * 1.44269504088896341f;
  }
  a.lse2[((size_t)s * LH + lh) * a.rows_pad + row] = l2;
}

template <int D, int RG, bool C>
hipError_t launch_passes_c(const SaliencyArgs& a, SaliencyMode mode, hipStream_t st) {
  const int LH = a.L * a.Hkv;
  const unsigned grid = (unsigned)LH * (unsigned)a.total_chunks;
  if (mode == SaliencyMode::kBoth && a.unit_cnt) {
    const hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(a.unit_cnt), 0u, a.S * LH, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((saliency_fused_kernel<D, RG, C>), dim3(2 * grid), dim3(kThreads), 0, st, a);
    return hipGetLastError();
  }
  if (mode != SaliencyMode::kFromLse) {
    hipLaunchKernelGGL((saliency_kernel<D, RG, 1, C>), dim3(grid), dim3(kThreads), 0, st, a);
    hipLaunchKernelGGL(lse_combine_kernel, dim3(a.S * LH), dim3(kCombineThreads), 0, st, a);
  } else {
    hipLaunchKernelGGL(lse_import_kernel, dim3(a.S * LH), dim3(a.rows_pad), 0, st, a);
  }
  if (mode != SaliencyMode::kLseOnly)
    hipLaunchKernelGGL((saliency_kernel<D, RG, 2, C>), dim3(grid), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

template <int D, int RG>
hipError_t launch_passes(const SaliencyArgs& a, SaliencyMode mode, hipStream_t st) {
  return a.causal ? launch_passes_c<D, RG, true>(a, mode, st)
                  : launch_passes_c<D, RG, false>(a, mode, st);
}

}  // namespace

int saliency_rows_pad(int R) { return R <= 64 ? 64 : (R <= 128 ? 128 : 256); }
int saliency_tile_keys(int R) { return 32 * (4 / (saliency_rows_pad(R) / 64)); }

hipError_t launch_saliency(const SaliencyArgs& a, int d, SaliencyMode mode, hipStream_t st) {
  if (a.total_chunks == 0) {  // no keys at all: every exported row LSE is -inf
    if (mode == SaliencyMode::kLseOnly)
      hipLaunchKernelGGL(lse_combine_kernel, dim3(a.S * a.L * a.Hkv), dim3(kCombineThreads), 0, st,
                         a);
    return hipGetLastError();
  }
  const int rg = a.rows_pad / 64;
  if (d == 128) {
    if (rg == 1) return launch_passes<128, 1>(a, mode, st);
    if (rg == 2) return launch_passes<128, 2>(a, mode, st);
    return launch_passes<128, 4>(a, mode, st);
  }
  if (rg == 1) return launch_passes<64, 1>(a, mode, st);
  if (rg == 2) return launch_passes<64, 2>(a, mode, st);
  return launch_passes<64, 4>(a, mode, st);
}

}  // namespace stepkv
