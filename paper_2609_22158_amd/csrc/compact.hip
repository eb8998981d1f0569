// K/V compaction (eq. problem): C_hat = C_prot || C_traj[K], a bit-exact
// gather of whole key/value rows into a dense retained cache, in position
// order. One 16-byte piece per lane, whole rows per lane group, non-temporal
// loads and stores (every byte is touched once).
#include "common.h"
#include "internal.h"

namespace stepkv {
namespace {

constexpr int kThreads = 256;
constexpr int kRowsPerBlock = 64;

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(kThreads) void compact_kernel(CompactArgs a) {
  constexpr int kLanesPerRow = 2 * D / 16;
  constexpr int kRowsPerPass = kThreads / kLanesPerRow;
  const int nb = (a.out_rows + kRowsPerBlock - 1) / kRowsPerBlock;
  const int lh = blockIdx.x / nb, rb = blockIdx.x - lh * nb;
  const int total = min(a.out_rows, a.cu_retained[a.S]);
  const int r_end = min(total, (rb + 1) * kRowsPerBlock);
  const int sub = threadIdx.x / kLanesPerRow, piece = threadIdx.x % kLanesPerRow;
  const size_t in_head = (size_t)lh * a.ntot;
  const size_t out_head = (size_t)lh * a.out_rows;
  for (int o = rb * kRowsPerBlock + sub; o < r_end; o += kRowsPerPass) {
    const int s = segment_of(a.cu_retained, a.S, o);
    const int j = o - a.cu_retained[s];
    const int seq0 = a.cu_seqlens[s], ns = a.cu_seqlens[s + 1] - seq0;
    if (j < 0 || j >= ns) continue;
    const int pos = a.idx[(a.shared_idx ? 0 : in_head) + seq0 + j];
    if (pos < 0 || pos >= ns) continue;  // not a valid position: row left untouched
    const size_t src = (in_head + seq0 + pos) * (size_t)D;
    const size_t dst = (out_head + o) * (size_t)D;
    const u32x4_t kv = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.k + src) + piece);
    const u32x4_t vv = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.v + src) + piece);
    __builtin_nontemporal_store(kv, reinterpret_cast<u32x4_t*>(a.k_out + dst) + piece);
    __builtin_nontemporal_store(vv, reinterpret_cast<u32x4_t*>(a.v_out + dst) + piece);
  }
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, hipStream_t st) {
  if (a.out_rows <= 0 || a.LH == 0) return hipSuccess;
  const unsigned nb = (unsigned)((a.out_rows + kRowsPerBlock - 1) / kRowsPerBlock);
  const dim3 grid((unsigned)a.LH * nb);
  if (a.d == 128)
    hipLaunchKernelGGL(compact_kernel<128>, grid, dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(compact_kernel<64>, grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace stepkv
