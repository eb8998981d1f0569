// Kernel launch interface between the C ABI layer (api.cpp) and the HIP
// kernels. Every launcher enqueues on the given stream and returns the
// hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace stepkv {

// ---------------------------------------------------------------- saliency
struct SaliencyArgs {
  const uint16_t* q;         // bf16 [L][S][W][Hq][d]
  const uint16_t* k;         // bf16 [L*Hkv][Ntot][d]
  const int32_t* cu_seqlens; // [S+1]
  float2* partial;           // [L*Hkv][total_chunks][rows_pad] (log2 max, sum)
  float* lse2;               // [S][L*Hkv][rows_pad] log2-domain log-sum-exp
  float* sal;                // [L*Hkv][Ntot] A_i
  const float* lse_in;       // [L][S][W][Hq] natural-log row LSE given by the caller
  float* lse_out;            // [L][S][W][Hq] natural-log row LSE exported (or null)
  int L, S, W, Hq, Hkv, G;
  int row0;      // first window row (w * G + g) of this launch's row group
  int R;         // window rows in the group (at most 256)
  int rows_pad;  // R padded to 64, 128 or 256
  int accumulate;  // nonzero: the column-sum sweep adds to sal (groups after the first)
  int ntot, chunk, total_chunks;
  int causal;  // nonzero: window slot w sees keys 0 .. N_s - W + w only
  float c;     // softmax scale * log2(e)
  // both sweeps in one launch (saliency_fused_kernel) when set: per (sequence,
  // head) counters [S][L*Hkv], cleared by the launcher; lag = row-LSE items
  // ahead of the column-sum items
  int* unit_cnt;
  int lag;
  uint32_t* status;  // device status word (STEPKV_FLAG_*) or null
  // Batches of at most kArgSeqs sequences also pass cu_seqlens and each
  // sequence's first chunk (at this launch's chunk size) by value: a workgroup
  // then finds its chunk with scalar loads of its arguments, where a read of
  // cu_seqlens would queue behind the K stream of the compute unit's other
  // workgroup. Entries past S: seq_first = Ntot, chunk_first = INT_MAX.
  static constexpr int kArgSeqs = 32;
  int seq_first[kArgSeqs + 1];
  int chunk_first[kArgSeqs + 1];
};

// Rows padded to whole row groups: 64, 128 or 256.
int saliency_rows_pad(int R);
// Key tile processed per iteration by one workgroup.
int saliency_tile_keys(int R);
// Which sweeps to run: both (A from Q and K alone), the first one only (row
// LSE, exported to lse_out), or the second one only (from lse_in).
enum class SaliencyMode { kBoth, kLseOnly, kFromLse };
hipError_t launch_saliency(const SaliencyArgs& a, int d, SaliencyMode mode, hipStream_t st);

// ---------------------------------------------------------------- fuse
struct FuseArgs {
  const float* sal;          // [L*Hkv][Ntot]
  const int32_t* cu_seqlens; // [S+1]
  const int32_t* cu_steps;   // [S+1]
  const int32_t* step_ids;   // [Ntot]
  const uint8_t* prot;       // [Ntot]
  const float* util;         // [cu_steps[S]]
  float* scores;             // [L*Hkv][Ntot]
  void* stats;               // stepkv_step_stat [L*Hkv][cu_steps[S]] or null
  uint32_t* status;          // device status word (STEPKV_FLAG_*) or null
  int S, LH, ntot, total_steps, half, max_steps, max_len;
  int total_chunks;          // prio_chunks(): workgroups per row without statistics
  float alpha, beta;
};
// Chunks of 2048 positions over the sequences (the priority without statistics).
int prio_chunks(const int32_t* cu_seqlens_host, int S);
hipError_t launch_fuse(const FuseArgs& a, hipStream_t st);

// Shared-index priority without step statistics, over chunks of 256 positions.
struct SharedPrioArgs {
  const float* heads;        // [nheads][Ntot] per-head saliency of the last layers
  float* sal;                // [Ntot] summed saliency (written by the first kernel)
  float* cmax;               // [chunks] maximum pooled prunable value per chunk
  const int32_t* cu_seqlens; // [S+1]
  const int32_t* cu_steps;   // [S+1]
  const int32_t* step_ids;   // [Ntot]
  const uint8_t* prot;       // [Ntot]
  const float* util;         // [cu_steps[S]]
  float* scores;             // [Ntot]
  uint32_t* status;          // device status word (STEPKV_FLAG_*) or null
  int S, ntot, nheads, half;
  float alpha, beta;
};
int shared_chunks(const int32_t* cu_seqlens_host, int S);
hipError_t launch_shared_priority(const SharedPrioArgs& a, int chunks, hipStream_t st);
// out[i] = sum over h < heads of sal[h][i] (fp32, [heads][ntot] -> [ntot]).
hipError_t launch_sum_heads(const float* sal, int heads, int ntot, float* out, hipStream_t st);

// ---------------------------------------------------------------- select
struct SelectArgs {
  const float* scores;       // [L*Hkv][Ntot]
  const uint8_t* prot;       // [Ntot]
  const int32_t* step_ids;   // [Ntot]
  const int32_t* cu_seqlens; // [S+1]
  const int32_t* cu_steps;   // [S+1]
  const int32_t* budgets;    // [S] or null
  int32_t* idx;              // [L*Hkv][Ntot]
  int32_t* cu_retained;      // [S+1]
  int32_t* kept;             // [L*Hkv][cu_steps[S]] or null
  int S, LH, ntot, total_steps, budget, max_len;
};
hipError_t launch_select(const SelectArgs& a, hipStream_t st);

// ---------------------------------------------------------------- compact
struct CompactArgs {
  const uint16_t* k;         // bf16 [L*Hkv][Ntot][d]
  const uint16_t* v;
  const int32_t* idx;        // [L*Hkv][Ntot], or [Ntot] shared by every head
  const int32_t* cu_seqlens; // [S+1]
  const int32_t* cu_retained;// [S+1]
  uint16_t* k_out;           // bf16 [L*Hkv][out_rows][d]
  uint16_t* v_out;
  uint32_t* status;          // device status word (STEPKV_FLAG_*) or null
  int S, LH, ntot, out_rows, d;
  int shared_idx;            // nonzero: one idx row for every (layer, KV head)
};
hipError_t launch_compact(const CompactArgs& a, hipStream_t st);

// HBM ceiling probe: read (copy = 0) or copy `bytes` (a multiple of 16) with
// the compaction's access width; a read writes at most one word per block of
// 256 threads to dst.
hipError_t launch_probe(const void* src, void* dst, size_t bytes, int copy, hipStream_t st);

// p[0 .. n) = v on the stream (a kernel, not a memset, so that it can sit in
// a captured graph).
hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int n, hipStream_t st);

// The static device scratch of stepkv_score_noalloc (STEPKV_STATIC_SCRATCH_BYTES):
// its address on the current device, looked up on the first call per device.
constexpr size_t kStaticScratchBytes = size_t(128) << 20;
hipError_t static_scratch(void** ptr);

// Device status bits (the STEPKV_FLAG_* values of stepkv.h).
constexpr uint32_t kFlagStepId = 1u, kFlagNonFinite = 2u, kFlagOutRows = 4u, kFlagSync = 8u;

// ---------------------------------------------------------------- decode check
struct DecodeArgs {
  const uint16_t* q;         // bf16 [L][S][Hq][d]
  const uint16_t* k;         // bf16 [L*Hkv][out_rows][d]
  const uint16_t* v;
  const int32_t* cu_retained;// [S+1]
  float* out;                // [L][S][Hq][d]
  const int32_t* cu_seqlens; // [S+1]
  float* partial;            // workspace: [L*Hkv][total_splits][G][d+2] (o, m, z)
  uint32_t* status;          // device status word (STEPKV_FLAG_*) or null
  int L, S, Hq, Hkv, G, d, out_rows, total_splits;
  int split_rows;            // retained rows per workgroup of the split kernel
  float scale;
};
// Rows per split for this cache size (512 or 1024).
int decode_split_rows(int L, int Hkv, int out_rows);
// Row splits of the split kernel (a host-side bound) for these sequence
// lengths, out_rows and rows per split.
int decode_total_splits(const int32_t* cu_seqlens_host, int S, int out_rows, int split_rows);
// Floats of partial state the launch needs (0 for groups above 16 heads).
size_t decode_partial_floats(const DecodeArgs& a);
hipError_t launch_decode(const DecodeArgs& a, hipStream_t st);

// Issue-rate probe: `blocks` workgroups of 256 threads, `iters` loops of four
// 32x32x16 bf16 MFMAs, alone (mix 0) or with the saliency sweeps' vector work
// for two score elements per MFMA (mix 1); one float per thread to sink.
hipError_t launch_issue_probe(int mix, int blocks, int iters, float* sink, hipStream_t st);

}  // namespace stepkv
