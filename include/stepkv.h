/*
 * stepkv.h - C ABI of the StepKV compression pass on AMD Instinct MI355X (gfx950).
 *
 * Paper: "StepKV: Step-Aware KV Cache Compression for LLM Agents".
 *
 * At a post-step pruning boundary (Sec. 3) the KV cache of every sequence is
 * C = C_prot || C_traj. The pass scores every cached token of every layer and
 * KV head, keeps the protected tokens plus the top-B prunable ones, and
 * rewrites the cache densely (eq. problem):
 *
 *   stepkv_score    window saliency T_i fused with step utility S_k into the
 *                   retention priority P_i = alpha*T_i + beta*S_k
 *                   (Sec. 5.2, eq. token-priority); it is the composition of
 *                   stepkv_saliency (the attention sweeps over K) and
 *                   stepkv_priority (pooling, normalisation, fusion).
 *                   stepkv_score_from_lse takes the window rows' log-sum-exps
 *                   from the caller's prefill (App. C.2) and sweeps K once.
 *   stepkv_select   global top-B ranking per (sequence, layer, KV head)
 *                   (Sec. 5.2 last paragraph; Algorithm 1 phase 3)
 *   stepkv_compact  C_hat = C_prot || C_traj[K] (eq. problem)
 *   stepkv_*_shared the same three steps with one ranking per sequence from
 *                   the last layers' saliency and one retained set for every
 *                   layer and head (App. D; Sec. 5.2)
 *
 * Host-only helpers implement the budget rule B_t = max(1, floor(rho N_t))
 * (eq. problem) and the step-utility update of Algorithm 1 phases 1-2
 * (eq. reward, eq. reuse, eq. step-score).
 *
 * Conventions for every call:
 *  - Tensor pointers are DEVICE pointers unless the name ends in _host. The
 *    caller owns every buffer; the library never allocates device memory and
 *    keeps no global state, so calls are re-entrant given distinct workspaces.
 *  - Device work is enqueued on `stream` (a hipStream_t; NULL = default
 *    stream) and is asynchronous: a return of STEPKV_OK means validation
 *    passed and every kernel was launched.
 *  - bf16 tensors hold raw bfloat16 values (2 bytes each).
 *  - Arguments are validated on the host before anything is launched; a
 *    failed validation returns an error code and launches nothing.
 *  - Outputs do not overlap inputs. Where a call takes both, scores and
 *    saliency are checked: overlapping ones are EINVAL.
 *  - No C++ exception crosses this interface.
 *  - Conditions only the device can see (a step id out of range, a
 *    non-finite input, rows past out_rows) are reported through the
 *    problem's optional status word (stepkv_problem.status,
 *    stepkv_status_read), not through return codes.
 *
 * Layouts (L layers, S sequences, Hq query heads, Hkv KV heads, G = Hq/Hkv,
 * d head dim, W window length, Ntot = cu_seqlens[S]):
 *  q_win        bf16  [L][S][W][Hq][d]   last W queries of every sequence
 *  lse_win      fp32  [L][S][W][Hq]      natural-log row log-sum-exp of them
 *  k, v         bf16  [L][Hkv][Ntot][d]  sequences concatenated along Ntot
 *  step_ids     int32 [Ntot]             step index local to the sequence
 *  protected    uint8 [Ntot]             nonzero = protected (never pruned)
 *  step_utility fp32  [cu_steps[S]]      S_k of sequence s at cu_steps[s] + k
 *  scores       fp32  [L][Hkv][Ntot]     P_i (protected tokens: -inf)
 *  saliency     fp32  [L][Hkv][Ntot]     A_i, the raw window saliency
 *  idx          int32 [L][Hkv][Ntot]     retained positions of sequence s
 *                                        (local, ascending) at offset
 *                                        cu_seqlens[s] of every (l, h) row
 *  cu_retained  int32 [S+1]              prefix sums of retained rows per
 *                                        sequence (same for every (l, h))
 *  k_out, v_out bf16  [L][Hkv][out_rows][d]  compacted cache; sequence s
 *                                        occupies rows cu_retained[s] ...
 */
#ifndef STEPKV_H_
#define STEPKV_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- errors */
#define STEPKV_OK 0
#define STEPKV_EINVAL (-1)       /* null pointer, bad shape or parameter */
#define STEPKV_EUNSUPPORTED (-2) /* valid but outside this build's limits */
#define STEPKV_EWORKSPACE (-3)   /* workspace missing or too small */
#define STEPKV_EHIP (-4)         /* a HIP launch or runtime call failed */
#define STEPKV_ESCRATCH (-5)     /* the problem needs more than the static scratch */

/* Limits of this build (STEPKV_EUNSUPPORTED beyond them). */
#define STEPKV_MAX_WINDOW_ROWS 2048  /* W * G (above 256: one pair of sweeps per 256 rows) */
#define STEPKV_MAX_POOL_KERNEL 63    /* odd pooling window */
#define STEPKV_MAX_STEPS_STATS 4096  /* steps per sequence when stats are requested */
#define STEPKV_CUE_CAP 64            /* evidence cues per text field (App. D) */

/* Conditions the kernels detect on the device (stepkv_problem.status). None
 * stops a call: each result stays defined as the call's text says. */
#define STEPKV_FLAG_STEP_ID 1u   /* a prunable token's step id lies outside [0, n_steps_s):
                                    it took utility 0 (priority, score calls) */
#define STEPKV_FLAG_NONFINITE 2u /* a prunable token's saliency or step utility was NaN or
                                    infinite (NaN or inf in q_win, k, lse_win or
                                    step_utility); its priority is not finite */
#define STEPKV_FLAG_OUT_ROWS 4u  /* cu_retained[S] exceeded out_rows: rows at or past
                                    out_rows were not written (compact) or read (decode) */
#define STEPKV_FLAG_SYNC 8u      /* a column-sum workgroup of the one-launch saliency
                                    sweeps stopped waiting for its (sequence, head)'s row
                                    LSEs after its poll bound: that head's saliency and
                                    scores are not valid (not expected to occur) */

/* ---------------------------------------------------------------- types */
/* Shape of one compression problem: a batch of S sequences, all layers. */
typedef struct stepkv_problem {
  int32_t num_layers;   /* L >= 1 */
  int32_t num_q_heads;  /* Hq >= 1, a multiple of num_kv_heads */
  int32_t num_kv_heads; /* Hkv >= 1 */
  int32_t head_dim;     /* d: 64 or 128 */
  int32_t window;       /* W >= 1 observation-window queries */
  int32_t num_seqs;     /* S >= 1 */
  const int32_t* cu_seqlens_host; /* [S+1] host: 0 = cu[0] <= cu[1] <= ... (read at
                                     every call: it sizes the launches, and for S <= 32
                                     the saliency sweeps take its values as launch
                                     arguments; a captured graph keeps those) */
  const int32_t* cu_seqlens;      /* [S+1] device copy of the same values */
  const int32_t* cu_steps_host;   /* [S+1] host: offsets into step_utility */
  const int32_t* cu_steps;        /* [S+1] device copy of the same values */
  /* Device status word (uint32 [1], caller-owned) or NULL. When set, the
   * kernels of every device call on this problem OR the STEPKV_FLAG_* bits of
   * the conditions they meet into it; nothing else writes it. The caller
   * zeroes it once (or through stepkv_status_read) and reads it back with
   * stepkv_status_read. Calls that may run at the same time share it. */
  uint32_t* status;
} stepkv_problem;

/* Method parameters; stepkv_params_default() fills the paper's defaults
 * (hyper-parameter table, App. D). */
typedef struct stepkv_params {
  float alpha;          /* token-saliency weight (0.2) */
  float beta;           /* step-utility weight (0.8) */
  int32_t pool_kernel;  /* odd 1-D average-pool window over A (7) */
  float scale;          /* softmax scale; <= 0 selects 1/sqrt(d) */
  /* step utility (Sec. 5.1) */
  float lambda_red;     /* redundancy penalty lambda (0.3) */
  float w_r, w_c;       /* completion / reuse weights (0.85, 0.15) */
  float r_min, r_max;   /* completion-score clip (-1, 2) */
  float s_max;          /* utility clip S_max (8) */
  float eta;            /* reuse update scale (1.5) */
  /* window visibility (0): 0 = every window row sees all N_s keys of its
   * sequence; nonzero = window slot w is the query at position N_s - W + w
   * and sees keys 0 .. N_s - W + w only, as in the causal attention of the
   * observation prefill that yields T_i (App. C.2). A row that sees no key
   * (N_s < W - w) contributes nothing. */
  int32_t causal_tail;
  /* schedule of the two saliency sweeps (0), a performance choice only (the
   * results agree to rounding): 0 = chosen per problem: both sweeps in one
   * launch, each key chunk's column sums about one round of workgroups after
   * its row LSEs so that K is read again from the Infinity Cache, when K
   * exceeds 192 MiB and there are at least twice as many chunks as resident
   * workgroups, otherwise one launch per sweep; 1 = one launch per sweep;
   * 2 = one launch. Calls given the row LSEs run one sweep either way. */
  int32_t saliency_schedule;
} stepkv_params;

/* Per-step statistics of one (layer, KV head, step), from stepkv_score:
 * over the step's prunable tokens, their count, the max of the normalised
 * saliency T_hat, and its sum in unsigned fixed point with 32 fractional bits
 * (sum = sum_q32 / 2^32), accumulated order-independently. */
typedef struct stepkv_step_stat {
  uint32_t count;
  float max_saliency;
  uint64_t sum_saliency_q32;
} stepkv_step_stat;

/* Step-utility state of one trajectory for the host update (Algorithm 1
 * phases 1-2). Arrays are caller-owned with room for `capacity` steps. */
typedef struct stepkv_step_state {
  int32_t capacity;  /* entries available in r and c */
  int32_t num_steps; /* t: completed steps so far (start at 0) */
  double* r;         /* completion score r_k (eq. reward) */
  double* c;         /* reuse accumulator c_k (eq. reuse) */
} stepkv_step_state;

/* ---------------------------------------------------------------- host helpers */
/* Fill the paper's default parameters (App. D hyper-parameter table) and the
 * 1-D pooling window 7. Never fails for a non-null pointer. */
void stepkv_params_default(stepkv_params* prm);

/* Static text for an error code. */
const char* stepkv_strerror(int code);

/* eq. problem: B = max(1, floor(rho * n_prunable)), rho in (0, 1].
 * Returns -1 for rho outside (0, 1] or n_prunable < 0. */
int64_t stepkv_budget_from_ratio(double rho, int64_t n_prunable);

/* eq. problem, with exactly min(B_s, N_pr,s) prunable tokens kept (Algorithm 1
 * output): the compacted rows of every sequence,
 *   R_s = P_s + min(B_s, N_s - P_s),  P_s = protected tokens of sequence s,
 * prefix-summed into cu_retained_host [S+1] (host); cu_retained_host[S] is
 * the out_rows that stepkv_compact needs. B_s is `budget`, or
 * max(1, budgets_host[s]) when budgets_host (host int32 [S]) is non-NULL:
 * the same rule, clamp included, as stepkv_select, whose cu_retained equals
 * this result. protected_host is the host copy of the protected mask, uint8
 * [cu_seqlens_host[S]] (nonzero = protected). Host only.
 * Errors: EINVAL for a null or bad problem, null protected_host or
 * cu_retained_host, budget < 1 without budgets_host, or a total beyond
 * INT32_MAX. */
int stepkv_retained_rows(const stepkv_problem* pb, const uint8_t* protected_host, int32_t budget,
                         const int32_t* budgets_host, int32_t* cu_retained_host);

/* Reads the problem's device status word (pb->status) after the work queued
 * on `stream` so far has finished (the call waits for the stream), into
 * *flags_host, and sets it to zero when `clear` is nonzero (on the stream,
 * waited for). The call synchronizes, so it does not belong inside a
 * captured HIP graph. Errors: EINVAL (null pb, pb->status or flags_host),
 * EHIP. */
int stepkv_status_read(const stepkv_problem* pb, uint32_t* flags_host, int32_t clear, void* stream);

/* Algorithm 1 phases 1-2 at the boundary after step t = state->num_steps + 1.
 * Phase 1: r_t = valid + gain - lambda*red (eq. reward; for the first step
 * gain = 1 and red = 0 by definition), c_t = 0. Phase 2: for k < t,
 * c_k += min(1, eta * obs_sim_prev[k]) (eq. reuse), where obs_sim_prev[k] is
 * sim(Obs_t, Obs_k) (host, t-1 entries; may be NULL when t = 1). Then writes
 * S_k = clip(w_r clip(r_k, r_min, r_max) + w_c ln(1 + c_k), 0, S_max)
 * (eq. step-score) for all k <= t into S_out (host, >= t floats).
 * Returns STEPKV_EINVAL for null state/params/S_out, a full state, or a
 * similarity outside [0, 1] or non-finite signal. O(t), host only. */
int stepkv_step_update(stepkv_step_state* state, float valid, float gain, float red,
                       const float* obs_sim_prev, const stepkv_params* prm, float* S_out);

/* ---------------------------------------------------------------- step signals from text
 * Sec. 5.1.1 (observation validity, evidence gain, action redundancy) and the
 * observation similarities of the reuse update (eq. reuse, Sec. 5.1.2),
 * computed on the host from each step's Thought, Action and Observation text.
 * The paper's sim is an overlap of at most STEPKV_CUE_CAP extracted evidence
 * cues per field (App. D); here:
 *  - a cue is a maximal run of ASCII letters and digits (other bytes, UTF-8
 *    included, separate cues), lowercased, of two or more bytes, and not a
 *    common English function word; a field keeps its distinct cues in order
 *    of first appearance, the first STEPKV_CUE_CAP;
 *  - sim(a, b) = |A & B| / |A | B| (0 when both are empty);
 *  - valid = 0 when the observation has no cue or starts (after ASCII
 *    whitespace, case-insensitively) with an error marker: "error",
 *    "exception", "traceback", "invalid", "failed", "failure", "no results",
 *    "not found", "timed out", "timeout";
 *  - gain_k = 1 - max_{u<k} sim(Th_k || Obs_k, Th_u || Obs_u), gain_1 = 1;
 *    red_k = max_{u<k} sim(Act_k, Act_u), red_1 = 0.
 * The trajectory's state is caller-owned host memory (8-byte aligned) of
 * stepkv_text_state_bytes(capacity) bytes; texts are (pointer, length) pairs
 * of bytes, not necessarily NUL-terminated. The outputs feed
 * stepkv_step_update for the same boundary. Host-only; O(t) per boundary. */

/* Bytes of host state for a trajectory of up to `capacity` steps (0 if < 1). */
size_t stepkv_text_state_bytes(int32_t capacity);

/* Initialise (or reset) a trajectory's text state. EINVAL: null or misaligned
 * state, capacity < 1 or bytes too small. */
int stepkv_text_state_init(void* state, size_t bytes, int32_t capacity);

/* Add step t (the t-th call since init): extract its cues, write valid, gain,
 * red and obs_sim_prev[k] = sim(Obs_t, Obs_k) for k < t (t floats; may be
 * NULL when t = 0). EINVAL: null outputs, an uninitialised or full state, a
 * negative length or a NULL text with a positive length. */
int stepkv_text_step(void* state, const char* thought, int64_t thought_len, const char* action,
                     int64_t action_len, const char* observation, int64_t observation_len,
                     float* valid, float* gain, float* red, float* obs_sim_prev);

/* The cues of one text as 64-bit FNV-1a hashes of their lowercased bytes, in
 * order of first appearance: cues[0 .. *count), *count <= STEPKV_CUE_CAP. */
int stepkv_text_cues(const char* text, int64_t text_len, uint64_t* cues, int32_t* count);

/* ---------------------------------------------------------------- device passes */
/* Bytes of device workspace stepkv_score needs for this problem (0 when the
 * problem is invalid). The workspace needs no initialisation and is
 * scratch between calls; 256-byte alignment is required. */
size_t stepkv_score_workspace_bytes(const stepkv_problem* pb);

/* Bytes of device workspace stepkv_saliency needs (0 when invalid); never
 * more than stepkv_score_workspace_bytes. Same rules. */
size_t stepkv_saliency_workspace_bytes(const stepkv_problem* pb);

/* Sec. 5.2, token saliency: the raw observation-window saliency
 *   A_i = sum_r softmax_i(scale * q_r . k_i)
 * of every token, for every (sequence, layer, KV head), written to saliency
 * fp32 [L][Hkv][Ntot]. Window rows r = w*G + g use query head h*G + g; the
 * softmax runs over the keys each row sees (all N_s keys, or the causal tail
 * of prm->causal_tail). Computed exactly (two sweeps over K: row
 * log-sum-exp, then column sums), fp32 accumulation of bf16 products. Window
 * rows (r = w * G + g) run in groups of 256, one pair of sweeps per group; the
 * column sums of a later group are added to the earlier groups' in order.
 * Errors: EINVAL (null pointers, bad problem or scale), EUNSUPPORTED (d not in
 * {64,128} or W*G > STEPKV_MAX_WINDOW_ROWS), EWORKSPACE, EHIP. */
int stepkv_saliency(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                    const void* k, float* saliency, void* workspace, size_t ws_bytes,
                    void* stream);

/* Row log-sum-exp of the window attention (the first of the two sweeps):
 *   lse_win[l][s][w][h*G+g] = ln sum_{i seen by row (w,g)} exp(scale * q . k_i)
 * natural log, fp32 [L][S][W][Hq]; -inf for a row that sees no key. This is
 * the quantity a prefill attention kernel reports per query row, so either
 * source can feed stepkv_saliency_from_lse. Workspace and errors as
 * stepkv_saliency. */
int stepkv_window_lse(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                      const void* k, float* lse_win, void* workspace, size_t ws_bytes,
                      void* stream);

/* App. C.2: the token saliency collected inside the observation prefill,
 * whose attention has already normalised every window row. Given each row's
 * natural-log log-sum-exp lse_win fp32 [L][S][W][Hq] over the keys it sees
 * (as stepkv_window_lse returns, or as the prefill's attention reports for
 * the last W query positions when prm->causal_tail is set), one sweep over K
 * gives
 *   A_i = sum_{r seeing i} exp(scale * q_r . k_i - lse_r)
 * written like stepkv_saliency. An lse of -inf marks a row that sees no key.
 * The result equals stepkv_saliency's to rounding when lse_win is exact;
 * otherwise each row's contribution scales by exp(exact - given).
 * Workspace and errors as stepkv_saliency. */
int stepkv_saliency_from_lse(const stepkv_problem* pb, const stepkv_params* prm,
                             const void* q_win, const void* k, const float* lse_win,
                             float* saliency, void* workspace, size_t ws_bytes, void* stream);

/* Sec. 5.2, eq. token-priority, from a saliency computed by stepkv_saliency:
 *   T_i = (1/k) sum_{|j-i| <= k/2} A_j [j prunable], zero padding, per sequence
 *   Th_i = T_i / max_{prunable} T  (0 when that max is 0)
 *   P_i  = alpha * Th_i + beta * S_{step_ids[i]};  protected: -inf
 * plus the optional per-step statistics (see stepkv_score). No workspace:
 * without statistics, and with more (sequence, layer, KV head) rows than
 * 256 or more than 4096 steps in a sequence, each row is spread over
 * workgroups of 2048 positions, which keep their partial maxima in the
 * scores row until they overwrite it.
 * Errors: EINVAL (also scores overlapping saliency), EUNSUPPORTED (pool
 * window, stats step count), EHIP. */
int stepkv_priority(const stepkv_problem* pb, const stepkv_params* prm, const float* saliency,
                    const int32_t* step_ids, const uint8_t* protected_mask,
                    const float* step_utility, float* scores, stepkv_step_stat* step_stats,
                    void* stream);

/* Sec. 5.2: token saliency and retention priority, for every (layer, KV head).
 * For each sequence s, layer l and KV head h, with window rows r = w*G + g
 * (query head h*G + g) and the N_s keys of s:
 *   A_i   = sum_r softmax_i(scale * q_r . k_i)      (all N_s keys visible)
 *   T_i   = (1/k) sum_{|j-i| <= k/2} A_j [j prunable], zero padding, per sequence
 *   Th_i  = T_i / max_{prunable} T  (0 when that max is 0)
 *   P_i   = alpha * Th_i + beta * S_{step_ids[i]}   (eq. token-priority)
 * Protected tokens get P = -inf. A step id outside [0, n_steps_s) contributes
 * utility 0 and is left out of step_stats.
 * Outputs: scores (required); saliency = A (optional, NULL to skip);
 * step_stats [L][Hkv][cu_steps[S]] (optional, NULL to skip).
 * Errors: EINVAL for null required pointers or a bad problem/params,
 * EUNSUPPORTED for d not in {64,128}, W*G > STEPKV_MAX_WINDOW_ROWS or a
 * pool window above STEPKV_MAX_POOL_KERNEL (or more than
 * STEPKV_MAX_STEPS_STATS steps in one sequence when step_stats is requested),
 * EWORKSPACE when ws_bytes < stepkv_score_workspace_bytes(pb), EHIP on launch
 * failure. Results are deterministic (fixed reduction orders). */
int stepkv_score(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                 const void* k, const int32_t* step_ids, const uint8_t* protected_mask,
                 const float* step_utility, float* scores, float* saliency,
                 stepkv_step_stat* step_stats, void* workspace, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): stepkv_score
 * with its workspace taken from a static device buffer of
 * STEPKV_STATIC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends. The call allocates nothing and calls no allocating
 * routine; the caller still passes every input and output, and `saliency`
 * (fp32 [L][Hkv][Ntot], the A buffer the sweeps write) is required here.
 * Same arguments, results and errors as stepkv_score otherwise, plus
 * STEPKV_ESCRATCH when the problem needs more than the buffer
 * (stepkv_saliency_workspace_bytes(pb) > STEPKV_STATIC_SCRATCH_BYTES), found
 * before anything is launched. The first call on a device looks the buffer's
 * address up (EHIP if that fails). Every call on one GPU shares its buffer,
 * which keeps the last call's contents (no part of it needs to start at
 * zero): calls that overlap on one GPU, on different streams or threads,
 * race and must be ordered by the caller. */
#define STEPKV_STATIC_SCRATCH_BYTES ((size_t)128 << 20)
int stepkv_score_noalloc(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                         const void* k, const int32_t* step_ids, const uint8_t* protected_mask,
                         const float* step_utility, float* scores, float* saliency,
                         stepkv_step_stat* step_stats, void* stream);

/* stepkv_score with the saliency taken from given row log-sum-exps
 * (stepkv_saliency_from_lse, one sweep over K) instead of both sweeps.
 * Same outputs, workspace size and errors as stepkv_score. */
int stepkv_score_from_lse(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                          const void* k, const float* lse_win, const int32_t* step_ids,
                          const uint8_t* protected_mask, const float* step_utility,
                          float* scores, float* saliency, stepkv_step_stat* step_stats,
                          void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------- shared-index mode
 * The paper's own setting: token saliency from the last 3 layers (App. D,
 * hyper-parameter table) and one global ranking of each sequence's tokens
 * (Sec. 5.2), so that a single retained set indexes the cache of every layer
 * and KV head. Sequence-level outputs have one row per sequence:
 *   scores, saliency fp32 [Ntot]; idx int32 [Ntot]; step_stats and
 *   kept_per_step [cu_steps[S]].
 */

/* Bytes of device workspace stepkv_score_shared needs (0 when invalid). */
size_t stepkv_score_shared_workspace_bytes(const stepkv_problem* pb, int32_t last_layers);

/* Shared-index scoring. With n = min(last_layers, L) and layers L-n .. L-1:
 *   A_i  = sum over those layers l and KV heads h of A_i(l, h)
 *          (stepkv_saliency's A; from lse_win as in stepkv_saliency_from_lse
 *          when lse_win, fp32 [L][S][W][Hq], is non-NULL)
 *   T_i, Th_i, P_i as in stepkv_score, once per sequence.
 * scores (required) and saliency (= the summed A, optional) are fp32 [Ntot];
 * step_stats is [cu_steps[S]] (optional). Errors as stepkv_score, plus EINVAL
 * for last_layers < 1; EWORKSPACE below stepkv_score_shared_workspace_bytes. */
int stepkv_score_shared(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                        const void* k, const float* lse_win, int32_t last_layers,
                        const int32_t* step_ids, const uint8_t* protected_mask,
                        const float* step_utility, float* scores, float* saliency,
                        stepkv_step_stat* step_stats, void* workspace, size_t ws_bytes,
                        void* stream);

/* Shared-index selection: stepkv_select over one score row per sequence
 * (scores fp32 [Ntot]); writes idx int32 [Ntot] (ascending local positions of
 * sequence s at offset cu_seqlens[s]), cu_retained [S+1] and optionally
 * kept_per_step [cu_steps[S]]. Budgets as stepkv_select (e.g. B_t from
 * stepkv_budget_from_ratio per sequence via `budgets`). Errors as stepkv_select. */
int stepkv_select_shared(const stepkv_problem* pb, const float* scores,
                         const uint8_t* protected_mask, const int32_t* step_ids, int32_t budget,
                         const int32_t* budgets, int32_t* idx, int32_t* cu_retained,
                         int32_t* kept_per_step, void* stream);

/* Shared-index compaction (eq. problem with one retained set per sequence):
 * every (layer, KV head) row of k_out / v_out [L][Hkv][out_rows][d] gathers
 * the positions idx int32 [Ntot] of its own cache. Errors as stepkv_compact. */
int stepkv_compact_shared(const stepkv_problem* pb, const void* k, const void* v,
                          const int32_t* idx, const int32_t* cu_retained, int32_t out_rows,
                          void* k_out, void* v_out, void* stream);

/* Sec. 5.2 / Algorithm 1 phase 3 / eq. problem: for every (sequence, layer,
 * KV head), keep every protected token plus exactly min(B, N_pr) prunable
 * tokens, the first in the order (score descending, position ascending),
 * where NaN scores rank as -inf and -0.0 as +0.0. B is `budget`, or
 * budgets[s] when `budgets` (device int32 [S]) is non-NULL.
 * Writes idx (positions local to the sequence, ascending), cu_retained
 * (R_s = n_protected_s + min(B_s, N_pr_s) prefix-summed) and, optionally,
 * kept_per_step int32 [L][Hkv][cu_steps[S]] (retained prunable tokens per step).
 * Errors: EINVAL for null required pointers, a bad problem, budget < 1 (when
 * budgets is NULL); EHIP on launch failure. Budgets below 1 in `budgets` are
 * treated as 1. Deterministic. */
int stepkv_select(const stepkv_problem* pb, const float* scores, const uint8_t* protected_mask,
                  const int32_t* step_ids, int32_t budget, const int32_t* budgets, int32_t* idx,
                  int32_t* cu_retained, int32_t* kept_per_step, void* stream);

/* eq. problem: C_hat = C_prot || C_traj[K]. For every (l, h) and sequence s,
 * k_out[l][h][cu_retained[s] + j] = k[l][h][cu_seqlens[s] + idx[l][h][cu_seqlens[s] + j]]
 * for j < R_s, and likewise v. Rows at or beyond out_rows are not written
 * (cu_retained[S] gives the rows needed; stepkv_retained_rows computes it on
 * the host) and STEPKV_FLAG_OUT_ROWS is set in pb->status when rows were
 * dropped. A bit-exact copy; the outputs must
 * not overlap the inputs; k_out and v_out may be NULL when out_rows is 0.
 * Errors: EINVAL for null pointers, a bad problem or out_rows < 0; EHIP on
 * launch failure. */
int stepkv_compact(const stepkv_problem* pb, const void* k, const void* v, const int32_t* idx,
                   const int32_t* cu_retained, int32_t out_rows, void* k_out, void* v_out,
                   void* stream);

/* Bytes of device workspace stepkv_compress needs (0 when invalid): the score
 * workspace plus room for the scores and the retained positions, used when
 * the caller passes NULL for them. 256-byte alignment is required. */
size_t stepkv_compress_workspace_bytes(const stepkv_problem* pb);

/* The whole pass at one pruning boundary (Sec. 3; eq. problem; Algorithm 1
 * phase 3) as one call on one stream: stepkv_score (stepkv_score_from_lse
 * when lse_win is non-NULL), then stepkv_select, then stepkv_compact, with
 * the same arguments, layouts and results as those calls.
 *   scores  fp32 [L][Hkv][Ntot] or NULL (kept in the workspace)
 *   idx     int32 [L][Hkv][Ntot] or NULL (kept in the workspace)
 *   cu_retained int32 [S+1] (required)
 *   k_out, v_out bf16 [L][Hkv][out_rows][d]; out_rows from
 *           stepkv_retained_rows. A smaller out_rows drops the rows past it
 *           and sets STEPKV_FLAG_OUT_ROWS in pb->status (when set).
 * budget / budgets as stepkv_select (budgets: device int32 [S] or NULL).
 * Errors: those of the three calls (validated before anything is launched),
 * EWORKSPACE below stepkv_compress_workspace_bytes or misaligned. */
int stepkv_compress(const stepkv_problem* pb, const stepkv_params* prm, const void* q_win,
                    const void* k, const void* v, const float* lse_win, const int32_t* step_ids,
                    const uint8_t* protected_mask, const float* step_utility, int32_t budget,
                    const int32_t* budgets, float* scores, int32_t* idx, int32_t* cu_retained,
                    int32_t out_rows, void* k_out, void* v_out, void* workspace,
                    size_t ws_bytes, void* stream);

/* Bytes of device workspace stepkv_decode_attention needs (0 when invalid). */
size_t stepkv_decode_workspace_bytes(const stepkv_problem* pb, int32_t out_rows);

/* One decode step over a compacted cache (Sec. 3: the compacted cache serves
 * the next decoding steps): for every layer l, sequence s and query head hq
 * (KV head hq / G), out = softmax(scale * q . K_hat^T) V_hat over the R_s
 * rows of s (R_s from cu_retained, within out_rows). q_dec bf16 [L][S][Hq][d];
 * out fp32 [L][S][Hq][d] (zero for a sequence with no row); scale <= 0
 * selects 1/sqrt(d); k_hat and v_hat may be NULL when out_rows is 0. Rows at
 * or past out_rows are not read (STEPKV_FLAG_OUT_ROWS in pb->status when
 * cu_retained[S] exceeds out_rows; each sequence's range of cu_retained is
 * clamped to [0, out_rows)). Each KV head's rows are read once for its whole
 * query group (up to 16 heads; wider groups are served per query head),
 * split over workgroups of 512 rows, or 1024 rows when
 * L * Hkv * floor(out_rows / 1024) >= 1536. The workspace holds one partial
 * state (d + 2 floats) per (layer, KV head, split, head of the group), for
 * the splits min(sum_s ceil(min(N_s, out_rows) / split),
 * floor(out_rows / split) + S). Errors: EINVAL, EUNSUPPORTED (d), EWORKSPACE
 * (below stepkv_decode_workspace_bytes, or not 256-byte aligned), EHIP. */
int stepkv_decode_attention(const stepkv_problem* pb, const void* q_dec, const void* k_hat,
                            const void* v_hat, const int32_t* cu_retained, int32_t out_rows,
                            float scale, float* out, void* workspace, size_t ws_bytes,
                            void* stream);

/* ---------------------------------------------------------------- measurement
 * HBM ceiling probe (not part of the method): the bandwidth a plain streaming
 * kernel reaches on this device with the access width of the compaction (one
 * 16-byte non-temporal piece per thread), to set the measured kernels against.
 * copy = 0: read `bytes` from src (dst receives at most bytes / 4096 words);
 * copy != 0: copy `bytes` from src to dst (non-overlapping). bytes must be a
 * positive multiple of 16 and the pointers 16-byte aligned. Asynchronous on
 * `stream`. Errors: EINVAL, EHIP. */
int stepkv_bandwidth_probe(const void* src, void* dst, size_t bytes, int32_t copy, void* stream);

/* Issue-rate probe (not part of the method): the share of the matrix cores'
 * issue rate that the saliency sweeps' instruction mix leaves on this
 * device. Each wave of `blocks` workgroups of 256 threads loops `iters` times
 * over four independent v_mfma_f32_32x32x16_bf16 (32768 flops each); with
 * mix = 1 every MFMA is followed by the sweeps' vector work for two score
 * elements (a v_fma_f32, a v_exp_f32 and a v_add_f32 each, on independent
 * chains). Timing the call with mix 0 and with mix 1 on the same grid gives
 * the MFMA rate with and without that work. sink receives blocks * 256
 * floats (device memory, caller-owned). Asynchronous on `stream`.
 * Errors: EINVAL (mix not 0 or 1, blocks or iters below 1, null sink), EHIP. */
int stepkv_issue_probe(int32_t mix, int32_t blocks, int32_t iters, float* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* STEPKV_H_ */
