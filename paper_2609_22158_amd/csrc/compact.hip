// K/V compaction (eq. problem): C_hat = C_prot || C_traj[K], a bit-exact
// gather of whole key/value rows into a dense retained cache, in position
// order. One 16-byte piece per lane, whole rows per lane group, non-temporal
// loads and stores (every byte is touched once). One row per thread and many
// small blocks keep the most bytes in flight (one 16-byte piece per thread is
// also what a plain copy needs to approach the HBM ceiling on this part);
// with several rows per thread, all index loads go first, then all K/V loads.
// Each XCD works through a contiguous range of heads (6% faster than
// dealing consecutive row blocks to different XCDs).
#include "common.h"
#include "internal.h"

namespace stepkv {
namespace {

constexpr int kThreads = 256;
#ifndef STEPKV_COMPACT_PASSES
#define STEPKV_COMPACT_PASSES 1
#endif
constexpr int kPasses = STEPKV_COMPACT_PASSES;  // rows per thread

// Rows one block gathers: a row is 2d bytes, 16 per lane.
template <int D>
constexpr int rows_per_block() { return kThreads / (2 * D / 16) * kPasses; }

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// x[i] of an array that stays unchanged for the whole launch, read through the
// constant address space: with a wave-uniform index the load is a scalar one.
__device__ __forceinline__ int read_const(const int32_t* x, int i) {
  return ((const __attribute__((address_space(4))) int32_t*)x)[i];
}

template <int D>
__global__ __launch_bounds__(kThreads) void compact_kernel(CompactArgs a) {
  constexpr int kLanesPerRow = 2 * D / 16;
  constexpr int kRowsPerPass = kThreads / kLanesPerRow;
  constexpr int kRowsPerBlock = rows_per_block<D>();
  const int nb = (a.out_rows + kRowsPerBlock - 1) / kRowsPerBlock;
  // Workgroups are dealt to the 8 XCDs round-robin; XCD x takes the x-th
  // eighth of the (head, row block) list, so each XCD gathers from a
  // contiguous range of heads. The grid is padded to a multiple of 8.
  const int per = (int)(gridDim.x >> 3);
  const int bid = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (bid >= a.LH * nb) {
    // the first block past the gather (the grid always has one) reports rows
    // dropped past out_rows; the gather blocks carry no extra work for it
    if (bid == a.LH * nb && threadIdx.x == 0 && a.status && a.cu_retained[a.S] > a.out_rows)
      atomicOr(a.status, kFlagOutRows);
    return;
  }
  const int lh = bid / nb, rb = bid - lh * nb;
  const int total = min(a.out_rows, a.cu_retained[a.S]);
  const int sub = threadIdx.x / kLanesPerRow, piece = threadIdx.x % kLanesPerRow;
  const size_t in_head = (size_t)lh * a.ntot;
  const size_t out_head = (size_t)lh * a.out_rows;
  const int32_t* __restrict__ idx = a.idx + (a.shared_idx ? 0 : in_head);
  // 1. every row's source position (independent index loads). When the
  // block's rows all belong to one sequence (always, but at sequence
  // boundaries), that sequence and its bounds are found once, with scalar
  // loads: vector loads of them would queue behind the K/V loads of the other
  // blocks on the compute unit, and the index loads wait for them.
  const int o0 = rb * kRowsPerBlock;
  const int s0 = uniform(segment_of(a.cu_retained, a.S, max(min(o0, total - 1), 0)));
  const int r0 = read_const(a.cu_retained, s0), r1 = read_const(a.cu_retained, s0 + 1);
  const bool one_seq = o0 >= r0 && o0 + kRowsPerBlock <= r1;
  int src_row[kPasses];
  bool ok[kPasses];
  if (one_seq) {
    const int seq0 = read_const(a.cu_seqlens, s0), ns = read_const(a.cu_seqlens, s0 + 1) - seq0;
#pragma unroll
    for (int p = 0; p < kPasses; ++p) {
      const int o = o0 + p * kRowsPerPass + sub;
      const int j = o - r0;
      ok[p] = false;
      src_row[p] = 0;
      if (o < total && j < ns) {
        const int pos = idx[seq0 + j];
        ok[p] = pos >= 0 && pos < ns;  // not a valid position: row left untouched
        src_row[p] = ok[p] ? seq0 + pos : 0;
      }
    }
  } else {
#pragma unroll
    for (int p = 0; p < kPasses; ++p) {
      const int o = o0 + p * kRowsPerPass + sub;
      ok[p] = false;
      src_row[p] = 0;
      if (o < total) {
        const int s = segment_of(a.cu_retained, a.S, o);
        const int j = o - a.cu_retained[s];
        const int seq0 = a.cu_seqlens[s], ns = a.cu_seqlens[s + 1] - seq0;
        if (j < ns) {
          const int pos = idx[seq0 + j];
          ok[p] = pos >= 0 && pos < ns;
          src_row[p] = ok[p] ? seq0 + pos : 0;
        }
      }
    }
  }
  // 2. all K/V pieces in flight at once (row 0 of the head stands in for skipped rows)
  u32x4_t kv[kPasses], vv[kPasses];
#pragma unroll
  for (int p = 0; p < kPasses; ++p) {
    const size_t src = (in_head + src_row[p]) * (size_t)D;
    kv[p] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.k + src) + piece);
    vv[p] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.v + src) + piece);
  }
  // 3. the dense retained rows
#pragma unroll
  for (int p = 0; p < kPasses; ++p) {
    if (!ok[p]) continue;
    const int o = rb * kRowsPerBlock + p * kRowsPerPass + sub;
    const size_t dst = (out_head + o) * (size_t)D;
    __builtin_nontemporal_store(kv[p], reinterpret_cast<u32x4_t*>(a.k_out + dst) + piece);
    __builtin_nontemporal_store(vv[p], reinterpret_cast<u32x4_t*>(a.v_out + dst) + piece);
  }
}

__global__ void out_rows_check_kernel(const int32_t* __restrict__ cu_retained, int S,
                                      int out_rows, uint32_t* status) {
  if (threadIdx.x == 0 && cu_retained[S] > out_rows) atomicOr(status, kFlagOutRows);
}

// HBM ceiling probes: one 16-byte non-temporal piece per thread, the access
// width and pattern of the compaction, over n16 pieces. Read: every piece is
// loaded and folded into one word per block (so no load is dead). Copy: every
// piece is loaded and stored.
__global__ __launch_bounds__(kThreads) void probe_read_kernel(const u32x4_t* __restrict__ src,
                                                              size_t n16, uint32_t* __restrict__ out) {
  const size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
  uint32_t x = 0u;
  if (i < n16) {
    const u32x4_t v = __builtin_nontemporal_load(src + i);
    x = v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  x = (uint32_t)wave_sum_int((int)x);
  if ((threadIdx.x & (kWave - 1)) == 0 && x == 0x9e3779b9u) out[blockIdx.x] = x;  // rarely taken
}

__global__ __launch_bounds__(kThreads) void probe_copy_kernel(const u32x4_t* __restrict__ src,
                                                              u32x4_t* __restrict__ dst, size_t n16) {
  const size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n16) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

__global__ void fill_u32_kernel(uint32_t* __restrict__ p, uint32_t v, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

}  // namespace

hipError_t launch_probe(const void* src, void* dst, size_t bytes, int copy, hipStream_t st) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  const unsigned blocks = (unsigned)((n16 + kThreads - 1) / kThreads);
  if (copy)
    hipLaunchKernelGGL(probe_copy_kernel, dim3(blocks), dim3(kThreads), 0, st,
                       static_cast<const u32x4_t*>(src), static_cast<u32x4_t*>(dst), n16);
  else
    hipLaunchKernelGGL(probe_read_kernel, dim3(blocks), dim3(kThreads), 0, st,
                       static_cast<const u32x4_t*>(src), n16, static_cast<uint32_t*>(dst));
  return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_u32_kernel, dim3((n + 255) / 256), dim3(256), 0, st, p, v, n);
  return hipGetLastError();
}

hipError_t launch_compact(const CompactArgs& a, hipStream_t st) {
  // no tokens: nothing to gather (and no row 0 for skipped rows to stand on)
  if (a.out_rows <= 0 || a.LH == 0 || a.ntot == 0) {
    if (a.status && a.LH > 0)  // rows may still be needed past out_rows = 0
      hipLaunchKernelGGL(out_rows_check_kernel, dim3(1), dim3(64), 0, st, a.cu_retained, a.S,
                         a.out_rows, a.status);
    return hipGetLastError();
  }
  auto grid = [&](int rows_per_block) {  // a multiple of 8 (one eighth per XCD), one spare block
    const unsigned nb = (unsigned)((a.out_rows + rows_per_block - 1) / rows_per_block);
    return dim3(((unsigned)a.LH * nb + 1u + 7u) / 8u * 8u);
  };
  if (a.d == 128)
    hipLaunchKernelGGL(compact_kernel<128>, grid(rows_per_block<128>()), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(compact_kernel<64>, grid(rows_per_block<64>()), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace stepkv
