// C ABI of the StepKV compression pass: argument validation, launch planning,
// workspace layout, and the host-side step-utility update (Algorithm 1
// phases 1-2). Every device computation is a kernel launched from here.
#include "stepkv.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>

#include "internal.h"

using namespace stepkv;

namespace {

constexpr size_t kAlign = 256;
// Saliency work items: two resident workgroups on each of the 256 compute
// units, and a workgroup start (its Q fragments and first K tiles) costs
// about as long as six key tiles.
constexpr int kSalSlots = 2 * 256;
constexpr int kSalStartTiles = 6;
// Both saliency sweeps in one launch (stepkv_score and the shared-index
// scoring): a (sequence, head)'s column-sum chunks start about one round of
// resident workgroups after its row-LSE chunks, and the K that the row-LSE
// chunks in between read from HBM has to fit the 256 MB Infinity Cache
// beside it for the second read of the chunk to hit there. Shorter chunks
// keep that window smaller but start more workgroups; 192 MiB (about 2300-key
// chunks at d = 128) measured best on the 32k, 16k, ragged and last-query
// workloads.
constexpr int64_t kFusedReuseBytes = int64_t(192) << 20;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool monotone_from_zero(const int32_t* cu, int n) {
  if (cu[0] != 0) return false;
  for (int i = 0; i < n; ++i)
    if (cu[i + 1] < cu[i]) return false;
  return true;
}

int check_problem(const stepkv_problem* pb) {
  if (!pb) return STEPKV_EINVAL;
  if (pb->num_layers < 1 || pb->num_q_heads < 1 || pb->num_kv_heads < 1 || pb->window < 1 ||
      pb->num_seqs < 1 || pb->head_dim < 1)
    return STEPKV_EINVAL;
  if (pb->num_q_heads % pb->num_kv_heads != 0) return STEPKV_EINVAL;
  if (!pb->cu_seqlens_host || !pb->cu_seqlens || !pb->cu_steps_host || !pb->cu_steps)
    return STEPKV_EINVAL;
  if (!monotone_from_zero(pb->cu_seqlens_host, pb->num_seqs)) return STEPKV_EINVAL;
  if (!monotone_from_zero(pb->cu_steps_host, pb->num_seqs)) return STEPKV_EINVAL;
  if (pb->head_dim != 64 && pb->head_dim != 128) return STEPKV_EUNSUPPORTED;
  const int64_t lh = (int64_t)pb->num_layers * pb->num_kv_heads;
  if (lh * pb->num_seqs > std::numeric_limits<int32_t>::max()) return STEPKV_EUNSUPPORTED;
  return STEPKV_OK;
}

int window_rows(const stepkv_problem* pb) {
  return (int)std::min<int64_t>((int64_t)pb->window * (pb->num_q_heads / pb->num_kv_heads),
                                std::numeric_limits<int32_t>::max());
}

int max_seqlen(const stepkv_problem* pb) {
  int m = 0;
  for (int s = 0; s < pb->num_seqs; ++s)
    m = std::max(m, pb->cu_seqlens_host[s + 1] - pb->cu_seqlens_host[s]);
  return m;
}

struct SaliencyPlan {
  int R, rows_pad, chunk, total_chunks;
  // both sweeps in one launch: chunk, chunk count and row-LSE lead (items)
  int fused_chunk, fused_total_chunks, fused_lag;
  bool fused_pays;  // the schedule chosen per problem (stepkv_params.saliency_schedule 0)
};

// Window rows per pair of sweeps (the MFMA tiling holds at most 256).
constexpr int kRowGroup = 256;

SaliencyPlan plan_saliency(const stepkv_problem* pb) {
  SaliencyPlan p;
  p.R = window_rows(pb);
  p.rows_pad = saliency_rows_pad(std::min(p.R, kRowGroup));  // the first (widest) group
  const int64_t lh = (int64_t)pb->num_layers * pb->num_kv_heads;
  auto chunks_for = [&](int c) {
    int64_t t = 0;
    for (int s = 0; s < pb->num_seqs; ++s)
      t += (pb->cu_seqlens_host[s + 1] - pb->cu_seqlens_host[s] + c - 1) / c;
    return t;
  };
  // The chunk (a multiple of 128 keys, so every key tile divides it) with the
  // least estimated makespan, rounds of resident workgroups times the tiles
  // of one chunk plus a workgroup start; ties go to the longer chunk. Chunks
  // stop at 4096 keys: with several rounds the two workgroups of a compute
  // unit drift apart and each one's start hides under the other's sweep,
  // which a single round of simultaneous starts does not allow.
  const int tile = saliency_tile_keys(std::min(p.R, kRowGroup));
  p.chunk = 128;
  int64_t best = -1;
  for (int c = 128; c <= 4096; c += 128) {
    const int64_t rounds = (lh * chunks_for(c) + kSalSlots - 1) / kSalSlots;
    const int64_t cost = rounds * (c / tile + kSalStartTiles);
    if (best < 0 || cost <= best) {
      best = cost;
      p.chunk = c;
    }
  }
  p.total_chunks = (int)chunks_for(p.chunk);
  // One launch of both sweeps: the longest chunk (a multiple of 128 keys) whose
  // lead keeps the K read between a chunk's two sweeps within kFusedReuseBytes.
  // The lead is half the resident workgroups (the item order alternates the
  // sweeps) plus a sequence's chunks (its last row-LSE chunk comes that much
  // later) plus an eighth of the workgroups as margin; it is also at least a
  // sequence's chunk count, which orders every column-sum chunk after all
  // row-LSE chunks of its (sequence, head).
  auto most_chunks = [&](int c) {
    int m = 0;
    for (int s = 0; s < pb->num_seqs; ++s)
      m = std::max(m, (pb->cu_seqlens_host[s + 1] - pb->cu_seqlens_host[s] + c - 1) / c);
    return m;
  };
  auto lead = [&](int c) { return (int64_t)kSalSlots / 2 + most_chunks(c) + kSalSlots / 8; };
  p.fused_chunk = 128;
  for (int c = 128; c <= 4096; c += 128)
    if (lead(c) * c * 2 * pb->head_dim <= kFusedReuseBytes) p.fused_chunk = c;
  p.fused_total_chunks = (int)chunks_for(p.fused_chunk);
  p.fused_lag = (int)std::min<int64_t>(lead(p.fused_chunk), lh * p.fused_total_chunks);
  // One launch pays when K does not fit the reuse window anyway (otherwise the
  // second of two launches already finds it in the Infinity Cache) and there
  // are enough chunks for the row-LSE items to run a round ahead.
  const int64_t k_bytes = lh * (int64_t)pb->cu_seqlens_host[pb->num_seqs] * 2 * pb->head_dim;
  p.fused_pays = k_bytes > kFusedReuseBytes && lh * p.fused_total_chunks >= 2 * kSalSlots;
  return p;
}

struct WsLayout {
  size_t partial, lse, cnt, sal, total;
};

WsLayout layout(const stepkv_problem* pb, const SaliencyPlan& p) {
  const size_t lh = (size_t)pb->num_layers * pb->num_kv_heads;
  const size_t ntot = (size_t)pb->cu_seqlens_host[pb->num_seqs];
  WsLayout w;
  size_t off = 0;
  w.partial = off;  // sized for the longer chunk list of the two plans
  off = align_up(off + sizeof(float) * 2 * lh *
                           std::max(p.total_chunks, p.fused_total_chunks) * p.rows_pad);
  w.lse = off;
  off = align_up(off + sizeof(float) * pb->num_seqs * lh * p.rows_pad);
  w.cnt = off;  // per (sequence, head) counters of the one-launch sweeps
  off = align_up(off + sizeof(int32_t) * pb->num_seqs * lh);
  w.sal = off;
  off = align_up(off + sizeof(float) * lh * ntot);
  w.total = off;
  return w;
}

int hip_status(hipError_t e) { return e == hipSuccess ? STEPKV_OK : STEPKV_EHIP; }

double utility(double r, double c, const stepkv_params* p) {
  const double inner = std::min<double>(std::max<double>(r, p->r_min), p->r_max);
  const double v = (double)p->w_r * inner + (double)p->w_c * std::log1p(c);
  return std::min<double>(std::max(v, 0.0), p->s_max);
}

}  // namespace

extern "C" {

void stepkv_params_default(stepkv_params* p) {
  if (!p) return;
  p->alpha = 0.2f;
  p->beta = 0.8f;
  p->pool_kernel = 7;
  p->scale = 0.0f;
  p->lambda_red = 0.3f;
  p->w_r = 0.85f;
  p->w_c = 0.15f;
  p->r_min = -1.0f;
  p->r_max = 2.0f;
  p->s_max = 8.0f;
  p->eta = 1.5f;
  p->causal_tail = 0;
  p->saliency_schedule = 0;
}

const char* stepkv_strerror(int code) {
  switch (code) {
    case STEPKV_OK: return "ok";
    case STEPKV_EINVAL: return "invalid argument";
    case STEPKV_EUNSUPPORTED: return "unsupported shape or parameter";
    case STEPKV_EWORKSPACE: return "workspace missing or too small";
    case STEPKV_EHIP: return "HIP launch or runtime error";
    case STEPKV_ESCRATCH: return "problem needs more than the static scratch";
    default: return "unknown error";
  }
}

int64_t stepkv_budget_from_ratio(double rho, int64_t n_prunable) {
  if (!(rho > 0.0 && rho <= 1.0) || n_prunable < 0) return -1;
  const int64_t b = (int64_t)std::floor(rho * (double)n_prunable + 1e-9);
  return std::max<int64_t>(1, b);
}

int stepkv_retained_rows(const stepkv_problem* pb, const uint8_t* protected_host, int32_t budget,
                         const int32_t* budgets_host, int32_t* cu_retained_host) {
  if (!pb || pb->num_seqs < 1 || !pb->cu_seqlens_host || !protected_host || !cu_retained_host)
    return STEPKV_EINVAL;
  if (!monotone_from_zero(pb->cu_seqlens_host, pb->num_seqs)) return STEPKV_EINVAL;
  if (!budgets_host && budget < 1) return STEPKV_EINVAL;
  int64_t acc = 0;
  cu_retained_host[0] = 0;
  for (int s = 0; s < pb->num_seqs; ++s) {
    const int32_t a = pb->cu_seqlens_host[s], b = pb->cu_seqlens_host[s + 1];
    int64_t n_prot = 0;
    for (int32_t i = a; i < b; ++i) n_prot += protected_host[i] != 0;
    const int64_t n_pr = (b - a) - n_prot;
    const int64_t B = budgets_host ? std::max<int32_t>(1, budgets_host[s]) : budget;
    acc += n_prot + std::min(B, n_pr);
    if (acc > std::numeric_limits<int32_t>::max()) return STEPKV_EINVAL;
    cu_retained_host[s + 1] = (int32_t)acc;
  }
  return STEPKV_OK;
}

int stepkv_status_read(const stepkv_problem* pb, uint32_t* flags_host, int32_t clear,
                       void* stream) {
  if (!pb || !pb->status || !flags_host) return STEPKV_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint32_t v = 0u;
  if (hipMemcpyAsync(&v, pb->status, sizeof(v), hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return STEPKV_EHIP;
  if (clear) {
    if (launch_fill_u32(pb->status, 0u, 1, st) != hipSuccess || hipStreamSynchronize(st) != hipSuccess)
      return STEPKV_EHIP;
  }
  *flags_host = v;
  return STEPKV_OK;
}

int stepkv_step_update(stepkv_step_state* st, float valid, float gain, float red,
                       const float* obs_sim_prev, const stepkv_params* prm, float* S_out) {
  if (!st || !prm || !S_out || !st->r || !st->c) return STEPKV_EINVAL;
  const int t = st->num_steps;
  if (t < 0 || t >= st->capacity) return STEPKV_EINVAL;
  if (!std::isfinite(valid) || !std::isfinite(gain) || !std::isfinite(red)) return STEPKV_EINVAL;
  if (t > 0 && !obs_sim_prev) return STEPKV_EINVAL;
  for (int k = 0; k < t; ++k)
    if (!(obs_sim_prev[k] >= 0.0f && obs_sim_prev[k] <= 1.0f)) return STEPKV_EINVAL;
  // phase 1: new-step score (gain_1 = 1 and red_1 = 0 by definition)
  const double g = t == 0 ? 1.0 : (double)gain;
  const double rd = t == 0 ? 0.0 : (double)red;
  st->r[t] = (double)valid + g - (double)prm->lambda_red * rd;
  st->c[t] = 0.0;
  // phase 2: reuse credit for every earlier step
  for (int k = 0; k < t; ++k)
    st->c[k] += std::min(1.0, (double)prm->eta * (double)obs_sim_prev[k]);
  st->num_steps = t + 1;
  for (int k = 0; k <= t; ++k) S_out[k] = (float)utility(st->r[k], st->c[k], prm);
  return STEPKV_OK;
}

size_t stepkv_score_workspace_bytes(const stepkv_problem* pb) {
  if (check_problem(pb) != STEPKV_OK) return 0;
  return layout(pb, plan_saliency(pb)).total;
}

size_t stepkv_saliency_workspace_bytes(const stepkv_problem* pb) {
  if (check_problem(pb) != STEPKV_OK) return 0;
  return layout(pb, plan_saliency(pb)).sal;  // everything but the saliency buffer
}

}  // extern "C"

namespace {

int check_params(const stepkv_problem* pb, const stepkv_params* prm) {
  if (!prm) return STEPKV_EINVAL;
  if (!std::isfinite(prm->alpha) || !std::isfinite(prm->beta) || !std::isfinite(prm->scale))
    return STEPKV_EINVAL;
  if (prm->pool_kernel < 1 || prm->pool_kernel % 2 == 0) return STEPKV_EINVAL;
  if (prm->pool_kernel > STEPKV_MAX_POOL_KERNEL) return STEPKV_EUNSUPPORTED;
  if (prm->saliency_schedule < 0 || prm->saliency_schedule > 2) return STEPKV_EINVAL;
  if (window_rows(pb) > STEPKV_MAX_WINDOW_ROWS) return STEPKV_EUNSUPPORTED;
  return STEPKV_OK;
}

int max_steps_per_seq(const stepkv_problem* pb) {
  int m = 0;
  for (int s = 0; s < pb->num_seqs; ++s)
    m = std::max(m, pb->cu_steps_host[s + 1] - pb->cu_steps_host[s]);
  return m;
}

// Saliency sweeps into `sal` (or the row LSE into lse_out, or from lse_in),
// using workspace regions below layout().sal.
int run_saliency(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                 const void* k, float* sal, uint8_t* ws, hipStream_t st,
                 SaliencyMode mode = SaliencyMode::kBoth, const float* lse_in = nullptr,
                 float* lse_out = nullptr) {
  const SaliencyPlan plan = plan_saliency(pb);
  const WsLayout w = layout(pb, plan);
  const int d = pb->head_dim;
  SaliencyArgs sa;
  sa.q = static_cast<const uint16_t*>(q_win);
  sa.k = static_cast<const uint16_t*>(k);
  sa.cu_seqlens = pb->cu_seqlens;
  sa.partial = reinterpret_cast<float2*>(ws + w.partial);
  sa.lse2 = reinterpret_cast<float*>(ws + w.lse);
  sa.sal = sal;
  sa.lse_in = lse_in;
  sa.lse_out = lse_out;
  sa.causal = prm->causal_tail != 0;
  sa.L = pb->num_layers;
  sa.S = pb->num_seqs;
  sa.W = pb->window;
  sa.Hq = pb->num_q_heads;
  sa.Hkv = pb->num_kv_heads;
  sa.G = pb->num_q_heads / pb->num_kv_heads;
  sa.ntot = pb->cu_seqlens_host[pb->num_seqs];
  sa.status = pb->status;
  const bool fused = mode == SaliencyMode::kBoth &&
                     (prm->saliency_schedule == 0 ? plan.fused_pays : prm->saliency_schedule == 2);
  sa.chunk = fused ? plan.fused_chunk : plan.chunk;
  sa.total_chunks = fused ? plan.fused_total_chunks : plan.total_chunks;
  sa.unit_cnt = fused ? reinterpret_cast<int*>(ws + w.cnt) : nullptr;
  sa.lag = plan.fused_lag;
  // the chunk lookup's argument tables (used when S <= kArgSeqs)
  int64_t chunks_before = 0;
  for (int s = 0; s <= SaliencyArgs::kArgSeqs; ++s) {
    const bool in = s <= pb->num_seqs;
    sa.seq_first[s] = pb->cu_seqlens_host[in ? s : pb->num_seqs];
    sa.chunk_first[s] = in ? (int)chunks_before : std::numeric_limits<int>::max();
    if (s < pb->num_seqs)
      chunks_before +=
          (pb->cu_seqlens_host[s + 1] - pb->cu_seqlens_host[s] + sa.chunk - 1) / sa.chunk;
  }
  const double scale = prm->scale > 0.0f ? (double)prm->scale : 1.0 / std::sqrt((double)d);
  sa.c = (float)(scale * 1.4426950408889634);  // log2(e)
  // Window rows in groups of at most 256, one pair of sweeps per group: a
  // row's LSE needs only its own logits, and the column sums of the later
  // groups add to the first group's (the workspace regions are reused).
  for (int row0 = 0; row0 < plan.R; row0 += kRowGroup) {
    sa.row0 = row0;
    sa.R = std::min(kRowGroup, plan.R - row0);
    sa.rows_pad = saliency_rows_pad(sa.R);
    sa.accumulate = row0 > 0;
    const int rc = hip_status(launch_saliency(sa, d, mode, st));
    if (rc != STEPKV_OK) return rc;
  }
  return STEPKV_OK;
}

int run_priority(const stepkv_problem* pb, const stepkv_params* prm, const float* sal,
                 const int32_t* step_ids, const uint8_t* protected_mask, const float* util,
                 float* scores, stepkv_step_stat* stats, hipStream_t st) {
  FuseArgs fa;
  fa.sal = sal;
  fa.cu_seqlens = pb->cu_seqlens;
  fa.cu_steps = pb->cu_steps;
  fa.step_ids = step_ids;
  fa.prot = protected_mask;
  fa.util = util;
  fa.scores = scores;
  fa.stats = stats;
  fa.status = pb->status;
  fa.S = pb->num_seqs;
  fa.LH = pb->num_layers * pb->num_kv_heads;
  fa.ntot = pb->cu_seqlens_host[pb->num_seqs];
  fa.total_steps = pb->cu_steps_host[pb->num_seqs];
  fa.half = prm->pool_kernel / 2;
  fa.max_steps = std::max(max_steps_per_seq(pb), 1);
  fa.max_len = max_seqlen(pb);
  fa.total_chunks = prio_chunks(pb->cu_seqlens_host, pb->num_seqs);
  fa.alpha = prm->alpha;
  fa.beta = prm->beta;
  return hip_status(launch_fuse(fa, st));
}

// The priority reads the saliency around each position while other
// workgroups write scores (and keep partial results in the scores rows), so
// the two arrays of `rows` x Ntot floats must not share memory.
int check_priority_args(const stepkv_problem* pb, const int32_t* step_ids,
                        const uint8_t* protected_mask, const float* util, const float* scores,
                        const stepkv_step_stat* stats, const float* sal, size_t rows) {
  if (!step_ids || !protected_mask || !scores) return STEPKV_EINVAL;
  if (sal) {
    const uintptr_t n = sizeof(float) * rows * (size_t)pb->cu_seqlens_host[pb->num_seqs];
    const uintptr_t a = reinterpret_cast<uintptr_t>(sal), b = reinterpret_cast<uintptr_t>(scores);
    if (a < b + n && b < a + n) return STEPKV_EINVAL;
  }
  if (!util && pb->cu_steps_host[pb->num_seqs] > 0) return STEPKV_EINVAL;
  if (stats && max_steps_per_seq(pb) > STEPKV_MAX_STEPS_STATS) return STEPKV_EUNSUPPORTED;
  return STEPKV_OK;
}

bool aligned(const void* p) { return reinterpret_cast<uintptr_t>(p) % kAlign == 0; }

// Shared-index mode: the last n layers, as a problem of their own, plus the
// one-"head" view of the per-sequence ranking (one score row per sequence).
int shared_layers(const stepkv_problem* pb, int32_t last_layers) {
  return std::min<int>(std::max<int>(last_layers, 1), pb->num_layers);
}

stepkv_problem last_layers_view(const stepkv_problem* pb, int n) {
  stepkv_problem sub = *pb;
  sub.num_layers = n;
  return sub;
}

stepkv_problem one_head_view(const stepkv_problem* pb) {
  stepkv_problem one = *pb;
  one.num_layers = 1;
  one.num_q_heads = 1;
  one.num_kv_heads = 1;
  return one;
}

struct SharedLayout {
  size_t heads, shared, cmax, total;  // per-head saliency [n*Hkv][Ntot], summed A [Ntot],
                                      // chunk maxima of the multi-workgroup priority
};

SharedLayout shared_layout(const stepkv_problem* pb, int n) {
  const stepkv_problem sub = last_layers_view(pb, n);
  const size_t ntot = (size_t)pb->cu_seqlens_host[pb->num_seqs];
  SharedLayout w;
  w.heads = layout(&sub, plan_saliency(&sub)).sal;  // after the sweep workspace
  w.shared = align_up(w.heads + sizeof(float) * n * pb->num_kv_heads * ntot);
  w.cmax = align_up(w.shared + sizeof(float) * ntot);
  w.total = align_up(w.cmax + sizeof(float) * shared_chunks(pb->cu_seqlens_host, pb->num_seqs));
  return w;
}

// stepkv_compress: the score workspace (saliency buffer included), then the
// scores and the retained positions for callers that do not keep them.
struct CompressLayout {
  size_t scores, idx, total;
};

CompressLayout compress_layout(const stepkv_problem* pb) {
  const size_t entries = (size_t)pb->num_layers * pb->num_kv_heads *
                         (size_t)pb->cu_seqlens_host[pb->num_seqs];
  CompressLayout c;
  c.scores = layout(pb, plan_saliency(pb)).total;
  c.idx = align_up(c.scores + sizeof(float) * entries);
  c.total = align_up(c.idx + sizeof(int32_t) * entries);
  return c;
}

}  // namespace

extern "C" {

int stepkv_saliency(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                    const void* k, float* saliency, void* workspace, size_t ws_bytes,
                    void* stream) {
  int rc = check_problem(pb);
  if (rc == STEPKV_OK) rc = check_params(pb, prm);
  if (rc != STEPKV_OK) return rc;
  if (!q_win || !k || !saliency) return STEPKV_EINVAL;
  const WsLayout w = layout(pb, plan_saliency(pb));
  if (!workspace || ws_bytes < w.sal || !aligned(workspace)) return STEPKV_EWORKSPACE;
  if (pb->cu_seqlens_host[pb->num_seqs] == 0) return STEPKV_OK;
  return run_saliency(pb, prm, q_win, k, saliency, static_cast<uint8_t*>(workspace),
                      static_cast<hipStream_t>(stream));
}

int stepkv_priority(const stepkv_problem* pb, const stepkv_params* prm, const float* saliency,
                    const int32_t* step_ids, const uint8_t* protected_mask,
                    const float* step_utility, float* scores, stepkv_step_stat* step_stats,
                    void* stream) {
  int rc = check_problem(pb);
  if (rc == STEPKV_OK) rc = check_params(pb, prm);
  if (rc != STEPKV_OK) return rc;
  if (!saliency) return STEPKV_EINVAL;
  rc = check_priority_args(pb, step_ids, protected_mask, step_utility, scores, step_stats,
                           saliency, (size_t)pb->num_layers * pb->num_kv_heads);
  if (rc != STEPKV_OK) return rc;
  if (pb->cu_seqlens_host[pb->num_seqs] == 0) return STEPKV_OK;
  return run_priority(pb, prm, saliency, step_ids, protected_mask, step_utility, scores,
                      step_stats, static_cast<hipStream_t>(stream));
}

int stepkv_score(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                 const void* k, const int32_t* step_ids, const uint8_t* protected_mask,
                 const float* step_utility, float* scores, float* saliency,
                 stepkv_step_stat* step_stats, void* workspace, size_t ws_bytes, void* stream) {
  int rc = check_problem(pb);
  if (rc == STEPKV_OK) rc = check_params(pb, prm);
  if (rc != STEPKV_OK) return rc;
  if (!q_win || !k) return STEPKV_EINVAL;
  rc = check_priority_args(pb, step_ids, protected_mask, step_utility, scores, step_stats,
                           saliency, (size_t)pb->num_layers * pb->num_kv_heads);
  if (rc != STEPKV_OK) return rc;
  const WsLayout w = layout(pb, plan_saliency(pb));
  if (!workspace || ws_bytes < w.total || !aligned(workspace)) return STEPKV_EWORKSPACE;
  if (pb->cu_seqlens_host[pb->num_seqs] == 0) return STEPKV_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  float* sal = saliency ? saliency : reinterpret_cast<float*>(ws + w.sal);
  rc = run_saliency(pb, prm, q_win, k, sal, ws, st);
  if (rc != STEPKV_OK) return rc;
  return run_priority(pb, prm, sal, step_ids, protected_mask, step_utility, scores, step_stats,
                      st);
}

int stepkv_score_noalloc(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                         const void* k, const int32_t* step_ids, const uint8_t* protected_mask,
                         const float* step_utility, float* scores, float* saliency,
                         stepkv_step_stat* step_stats, void* stream) {
  static_assert(STEPKV_STATIC_SCRATCH_BYTES == kStaticScratchBytes, "one scratch size");
  int rc = check_problem(pb);
  if (rc == STEPKV_OK) rc = check_params(pb, prm);
  if (rc != STEPKV_OK) return rc;
  if (!q_win || !k || !saliency) return STEPKV_EINVAL;
  rc = check_priority_args(pb, step_ids, protected_mask, step_utility, scores, step_stats,
                           saliency, (size_t)pb->num_layers * pb->num_kv_heads);
  if (rc != STEPKV_OK) return rc;
  // the sweeps' workspace (everything but the saliency buffer, which the caller passes)
  if (layout(pb, plan_saliency(pb)).sal > kStaticScratchBytes) return STEPKV_ESCRATCH;
  if (pb->cu_seqlens_host[pb->num_seqs] == 0) return STEPKV_OK;
  void* ws = nullptr;
  if (static_scratch(&ws) != hipSuccess || !ws) return STEPKV_EHIP;
  hipStream_t st = static_cast<hipStream_t>(stream);
  rc = run_saliency(pb, prm, q_win, k, saliency, static_cast<uint8_t*>(ws), st);
  if (rc != STEPKV_OK) return rc;
  return run_priority(pb, prm, saliency, step_ids, protected_mask, step_utility, scores,
                      step_stats, st);
}

int stepkv_window_lse(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                      const void* k, float* lse_win, void* workspace, size_t ws_bytes,
                      void* stream) {
  int rc = check_problem(pb);
  if (rc == STEPKV_OK) rc = check_params(pb, prm);
  if (rc != STEPKV_OK) return rc;
  if (!q_win || !k || !lse_win) return STEPKV_EINVAL;
  const WsLayout w = layout(pb, plan_saliency(pb));
  if (!workspace || ws_bytes < w.sal || !aligned(workspace)) return STEPKV_EWORKSPACE;
  // runs even without keys: every row then sees none and gets -inf
  return run_saliency(pb, prm, q_win, k, nullptr, static_cast<uint8_t*>(workspace),
                      static_cast<hipStream_t>(stream), SaliencyMode::kLseOnly, nullptr, lse_win);
}

int stepkv_saliency_from_lse(const stepkv_problem* pb, const stepkv_params* prm,
                             const void* q_win, const void* k, const float* lse_win,
                             float* saliency, void* workspace, size_t ws_bytes, void* stream) {
  int rc = check_problem(pb);
  if (rc == STEPKV_OK) rc = check_params(pb, prm);
  if (rc != STEPKV_OK) return rc;
  if (!q_win || !k || !lse_win || !saliency) return STEPKV_EINVAL;
  const WsLayout w = layout(pb, plan_saliency(pb));
  if (!workspace || ws_bytes < w.sal || !aligned(workspace)) return STEPKV_EWORKSPACE;
  if (pb->cu_seqlens_host[pb->num_seqs] == 0) return STEPKV_OK;
  return run_saliency(pb, prm, q_win, k, saliency, static_cast<uint8_t*>(workspace),
                      static_cast<hipStream_t>(stream), SaliencyMode::kFromLse, lse_win);
}

int stepkv_score_from_lse(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                          const void* k, const float* lse_win, const int32_t* step_ids,
                          const uint8_t* protected_mask, const float* step_utility,
                          float* scores, float* saliency, stepkv_step_stat* step_stats,
                          void* workspace, size_t ws_bytes, void* stream) {
  int rc = check_problem(pb);
  if (rc == STEPKV_OK) rc = check_params(pb, prm);
  if (rc != STEPKV_OK) return rc;
  if (!q_win || !k || !lse_win) return STEPKV_EINVAL;
  rc = check_priority_args(pb, step_ids, protected_mask, step_utility, scores, step_stats,
                           saliency, (size_t)pb->num_layers * pb->num_kv_heads);
  if (rc != STEPKV_OK) return rc;
  const WsLayout w = layout(pb, plan_saliency(pb));
  if (!workspace || ws_bytes < w.total || !aligned(workspace)) return STEPKV_EWORKSPACE;
  if (pb->cu_seqlens_host[pb->num_seqs] == 0) return STEPKV_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  float* sal = saliency ? saliency : reinterpret_cast<float*>(ws + w.sal);
  rc = run_saliency(pb, prm, q_win, k, sal, ws, st, SaliencyMode::kFromLse, lse_win);
  if (rc != STEPKV_OK) return rc;
  return run_priority(pb, prm, sal, step_ids, protected_mask, step_utility, scores, step_stats,
                      st);
}

size_t stepkv_score_shared_workspace_bytes(const stepkv_problem* pb, int32_t last_layers) {
  if (check_problem(pb) != STEPKV_OK || last_layers < 1) return 0;
  return shared_layout(pb, shared_layers(pb, last_layers)).total;
}

int stepkv_score_shared(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                        const void* k, const float* lse_win, int32_t last_layers,
                        const int32_t* step_ids, const uint8_t* protected_mask,
                        const float* step_utility, float* scores, float* saliency,
                        stepkv_step_stat* step_stats, void* workspace, size_t ws_bytes,
                        void* stream) {
  int rc = check_problem(pb);
  if (rc == STEPKV_OK) rc = check_params(pb, prm);
  if (rc != STEPKV_OK) return rc;
  if (!q_win || !k || last_layers < 1) return STEPKV_EINVAL;
  rc = check_priority_args(pb, step_ids, protected_mask, step_utility, scores, step_stats,
                           saliency, 1);
  if (rc != STEPKV_OK) return rc;
  const int n = shared_layers(pb, last_layers);
  const SharedLayout w = shared_layout(pb, n);
  if (!workspace || ws_bytes < w.total || !aligned(workspace)) return STEPKV_EWORKSPACE;
  const int ntot = pb->cu_seqlens_host[pb->num_seqs];
  if (ntot == 0) return STEPKV_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  // the last n layers of q_win, k and lse_win
  const size_t first = (size_t)(pb->num_layers - n);
  const size_t q_layer = (size_t)pb->num_seqs * pb->window * pb->num_q_heads;  // rows per layer
  const uint16_t* q = static_cast<const uint16_t*>(q_win) + first * q_layer * pb->head_dim;
  const uint16_t* kk =
      static_cast<const uint16_t*>(k) + first * pb->num_kv_heads * (size_t)ntot * pb->head_dim;
  const float* lse = lse_win ? lse_win + first * q_layer : nullptr;
  const stepkv_problem sub = last_layers_view(pb, n);
  float* heads = reinterpret_cast<float*>(ws + w.heads);
  rc = run_saliency(&sub, prm, q, kk, heads, ws, st,
                    lse ? SaliencyMode::kFromLse : SaliencyMode::kBoth, lse);
  if (rc != STEPKV_OK) return rc;
  float* sal = saliency ? saliency : reinterpret_cast<float*>(ws + w.shared);
  if (!step_stats) {
    // one priority row per sequence, spread over chunks of positions
    SharedPrioArgs sa;
    sa.heads = heads;
    sa.sal = sal;
    sa.cmax = reinterpret_cast<float*>(ws + w.cmax);
    sa.cu_seqlens = pb->cu_seqlens;
    sa.cu_steps = pb->cu_steps;
    sa.step_ids = step_ids;
    sa.prot = protected_mask;
    sa.util = step_utility;
    sa.scores = scores;
    sa.status = pb->status;
    sa.S = pb->num_seqs;
    sa.ntot = ntot;
    sa.nheads = n * pb->num_kv_heads;
    sa.half = prm->pool_kernel / 2;
    sa.alpha = prm->alpha;
    sa.beta = prm->beta;
    return hip_status(
        launch_shared_priority(sa, shared_chunks(pb->cu_seqlens_host, pb->num_seqs), st));
  }
  rc = hip_status(launch_sum_heads(heads, n * pb->num_kv_heads, ntot, sal, st));
  if (rc != STEPKV_OK) return rc;
  const stepkv_problem one = one_head_view(pb);
  return run_priority(&one, prm, sal, step_ids, protected_mask, step_utility, scores, step_stats,
                      st);
}

int stepkv_select_shared(const stepkv_problem* pb, const float* scores,
                         const uint8_t* protected_mask, const int32_t* step_ids, int32_t budget,
                         const int32_t* budgets, int32_t* idx, int32_t* cu_retained,
                         int32_t* kept_per_step, void* stream) {
  const int rc = check_problem(pb);
  if (rc != STEPKV_OK) return rc;
  const stepkv_problem one = one_head_view(pb);
  return stepkv_select(&one, scores, protected_mask, step_ids, budget, budgets, idx, cu_retained,
                       kept_per_step, stream);
}

int stepkv_compact_shared(const stepkv_problem* pb, const void* k, const void* v,
                          const int32_t* idx, const int32_t* cu_retained, int32_t out_rows,
                          void* k_out, void* v_out, void* stream) {
  const int rc = check_problem(pb);
  if (rc != STEPKV_OK) return rc;
  if (!k || !v || !idx || !cu_retained || out_rows < 0) return STEPKV_EINVAL;
  if (out_rows > 0 && (!k_out || !v_out)) return STEPKV_EINVAL;  // NULL outputs hold 0 rows
  CompactArgs a;
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.idx = idx;
  a.cu_seqlens = pb->cu_seqlens;
  a.cu_retained = cu_retained;
  a.k_out = static_cast<uint16_t*>(k_out);
  a.v_out = static_cast<uint16_t*>(v_out);
  a.S = pb->num_seqs;
  a.LH = pb->num_layers * pb->num_kv_heads;
  a.ntot = pb->cu_seqlens_host[pb->num_seqs];
  a.out_rows = out_rows;
  a.d = pb->head_dim;
  a.shared_idx = 1;
  a.status = pb->status;
  return hip_status(launch_compact(a, static_cast<hipStream_t>(stream)));
}

int stepkv_select(const stepkv_problem* pb, const float* scores, const uint8_t* protected_mask,
                  const int32_t* step_ids, int32_t budget, const int32_t* budgets, int32_t* idx,
                  int32_t* cu_retained, int32_t* kept_per_step, void* stream) {
  const int rc = check_problem(pb);
  if (rc != STEPKV_OK) return rc;
  if (!scores || !protected_mask || !idx || !cu_retained) return STEPKV_EINVAL;
  if (kept_per_step && !step_ids) return STEPKV_EINVAL;
  if (!budgets && budget < 1) return STEPKV_EINVAL;
  SelectArgs a;
  a.scores = scores;
  a.prot = protected_mask;
  a.step_ids = step_ids;
  a.cu_seqlens = pb->cu_seqlens;
  a.cu_steps = pb->cu_steps;
  a.budgets = budgets;
  a.idx = idx;
  a.cu_retained = cu_retained;
  a.kept = kept_per_step;
  a.S = pb->num_seqs;
  a.LH = pb->num_layers * pb->num_kv_heads;
  a.ntot = pb->cu_seqlens_host[pb->num_seqs];
  a.total_steps = pb->cu_steps_host[pb->num_seqs];
  a.budget = std::max(budget, 1);
  a.max_len = max_seqlen(pb);
  return hip_status(launch_select(a, static_cast<hipStream_t>(stream)));
}

int stepkv_compact(const stepkv_problem* pb, const void* k, const void* v, const int32_t* idx,
                   const int32_t* cu_retained, int32_t out_rows, void* k_out, void* v_out,
                   void* stream) {
  const int rc = check_problem(pb);
  if (rc != STEPKV_OK) return rc;
  if (!k || !v || !idx || !cu_retained || out_rows < 0) return STEPKV_EINVAL;
  if (out_rows > 0 && (!k_out || !v_out)) return STEPKV_EINVAL;  // NULL outputs hold 0 rows
  CompactArgs a;
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.idx = idx;
  a.cu_seqlens = pb->cu_seqlens;
  a.cu_retained = cu_retained;
  a.k_out = static_cast<uint16_t*>(k_out);
  a.v_out = static_cast<uint16_t*>(v_out);
  a.S = pb->num_seqs;
  a.LH = pb->num_layers * pb->num_kv_heads;
  a.ntot = pb->cu_seqlens_host[pb->num_seqs];
  a.out_rows = out_rows;
  a.d = pb->head_dim;
  a.shared_idx = 0;
  a.status = pb->status;
  return hip_status(launch_compact(a, static_cast<hipStream_t>(stream)));
}

size_t stepkv_compress_workspace_bytes(const stepkv_problem* pb) {
  if (check_problem(pb) != STEPKV_OK) return 0;
  return compress_layout(pb).total;
}

int stepkv_compress(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                    const void* k, const void* v, const float* lse_win, const int32_t* step_ids,
                    const uint8_t* protected_mask, const float* step_utility, int32_t budget,
                    const int32_t* budgets, float* scores, int32_t* idx, int32_t* cu_retained,
                    int32_t out_rows, void* k_out, void* v_out, void* workspace,
                    size_t ws_bytes, void* stream) {
  // every argument of the three steps is validated before anything is launched
  int rc = check_problem(pb);
  if (rc == STEPKV_OK) rc = check_params(pb, prm);
  if (rc != STEPKV_OK) return rc;
  if (!q_win || !k || !v || !step_ids || !protected_mask || !cu_retained || out_rows < 0)
    return STEPKV_EINVAL;
  if (out_rows > 0 && (!k_out || !v_out)) return STEPKV_EINVAL;  // NULL outputs hold 0 rows
  if (!step_utility && pb->cu_steps_host[pb->num_seqs] > 0) return STEPKV_EINVAL;
  if (!budgets && budget < 1) return STEPKV_EINVAL;
  const CompressLayout cl = compress_layout(pb);
  if (!workspace || ws_bytes < cl.total || !aligned(workspace)) return STEPKV_EWORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  float* P = scores ? scores : reinterpret_cast<float*>(ws + cl.scores);
  int32_t* I = idx ? idx : reinterpret_cast<int32_t*>(ws + cl.idx);
  if (pb->cu_seqlens_host[pb->num_seqs] > 0) {
    float* sal = reinterpret_cast<float*>(ws + layout(pb, plan_saliency(pb)).sal);
    rc = run_saliency(pb, prm, q_win, k, sal, ws, st,
                      lse_win ? SaliencyMode::kFromLse : SaliencyMode::kBoth, lse_win);
    if (rc == STEPKV_OK)
      rc = run_priority(pb, prm, sal, step_ids, protected_mask, step_utility, P, nullptr, st);
    if (rc != STEPKV_OK) return rc;
  }
  rc = stepkv_select(pb, P, protected_mask, step_ids, budget, budgets, I, cu_retained, nullptr,
                     stream);
  if (rc != STEPKV_OK) return rc;
  return stepkv_compact(pb, k, v, I, cu_retained, out_rows, k_out, v_out, stream);
}

int stepkv_bandwidth_probe(const void* src, void* dst, size_t bytes, int32_t copy, void* stream) {
  if (!src || !dst || bytes == 0 || bytes % 16 != 0) return STEPKV_EINVAL;
  if (reinterpret_cast<uintptr_t>(src) % 16 != 0 || reinterpret_cast<uintptr_t>(dst) % 16 != 0)
    return STEPKV_EINVAL;
  return hip_status(launch_probe(src, dst, bytes, copy, static_cast<hipStream_t>(stream)));
}

int stepkv_issue_probe(int32_t mix, int32_t blocks, int32_t iters, float* sink, void* stream) {
  if ((mix != 0 && mix != 1) || blocks < 1 || iters < 1 || !sink) return STEPKV_EINVAL;
  return hip_status(launch_issue_probe(mix, blocks, iters, sink, static_cast<hipStream_t>(stream)));
}

size_t stepkv_decode_workspace_bytes(const stepkv_problem* pb, int32_t out_rows) {
  if (check_problem(pb) != STEPKV_OK || out_rows < 0) return 0;
  DecodeArgs a{};
  a.L = pb->num_layers;
  a.Hkv = pb->num_kv_heads;
  a.G = pb->num_q_heads / pb->num_kv_heads;
  a.d = pb->head_dim;
  a.split_rows = decode_split_rows(a.L, a.Hkv, out_rows);
  a.total_splits = decode_total_splits(pb->cu_seqlens_host, pb->num_seqs, out_rows, a.split_rows);
  return std::max<size_t>(sizeof(float) * decode_partial_floats(a), kAlign);
}

int stepkv_decode_attention(const stepkv_problem* pb, const void* q_dec, const void* k_hat,
                            const void* v_hat, const int32_t* cu_retained, int32_t out_rows,
                            float scale, float* out, void* workspace, size_t ws_bytes,
                            void* stream) {
  const int rc = check_problem(pb);
  if (rc != STEPKV_OK) return rc;
  if (!q_dec || !cu_retained || !out || out_rows < 0 || !std::isfinite(scale))
    return STEPKV_EINVAL;
  if (out_rows > 0 && (!k_hat || !v_hat)) return STEPKV_EINVAL;  // NULL caches hold 0 rows
  if (!workspace || ws_bytes < stepkv_decode_workspace_bytes(pb, out_rows) || !aligned(workspace))
    return STEPKV_EWORKSPACE;
  DecodeArgs a;
  a.q = static_cast<const uint16_t*>(q_dec);
  a.k = static_cast<const uint16_t*>(k_hat);
  a.v = static_cast<const uint16_t*>(v_hat);
  a.cu_retained = cu_retained;
  a.out = out;
  a.cu_seqlens = pb->cu_seqlens;
  a.partial = static_cast<float*>(workspace);
  a.status = pb->status;
  a.L = pb->num_layers;
  a.S = pb->num_seqs;
  a.Hq = pb->num_q_heads;
  a.Hkv = pb->num_kv_heads;
  a.G = pb->num_q_heads / pb->num_kv_heads;
  a.d = pb->head_dim;
  a.out_rows = out_rows;
  a.split_rows = decode_split_rows(a.L, a.Hkv, out_rows);
  a.total_splits = decode_total_splits(pb->cu_seqlens_host, pb->num_seqs, out_rows, a.split_rows);
  a.scale = scale > 0.0f ? scale : (float)(1.0 / std::sqrt((double)pb->head_dim));
  return hip_status(launch_decode(a, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
