/*
 * compress_demo.c - one StepKV compression pass driven through the C ABI
 * alone (HIP runtime for device memory, no Python), with self-checks.
 *
 * Two layers, GQA 8/2, d 128, W 16, two sequences of 700 and 301 tokens
 * with a 32-token protected prefix and 5 steps each, budget 64. Inputs are
 * seeded bf16 values from a 64-bit LCG. Checked on the host:
 *  - every (layer, head, sequence) saliency sums to W * G (each window row's
 *    softmax sums to one, Sec. 5.2);
 *  - protected tokens score -inf and prunable ones a finite P >= 0;
 *  - cu_retained[s+1] - cu_retained[s] = n_protected + min(B, N - n_protected)
 *    and each retained position list is ascending and holds the prefix;
 *  - every compacted K and V row equals the source row it names (bit-exact);
 *  - stepkv_retained_rows on the host gives the selection's cu_retained,
 *    stepkv_compress gives the three calls' outputs bit for bit, and the
 *    device status word stays clear.
 * Prints "ok" and returns 0, or names the first failed check and returns 1.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "stepkv.h"

enum { L = 2, HQ = 8, HKV = 2, D = 128, W = 16, S = 2, PROT = 32, STEPS = 5, BUDGET = 64 };
static const int32_t kLens[S] = {700, 301};

static uint64_t lcg = 0x9e3779b97f4a7c15ull;
static float next_uniform(void) { /* in [-1, 1) */
  lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
  return (float)((double)(lcg >> 11) * (1.0 / 9007199254740992.0)) * 2.0f - 1.0f;
}
static uint16_t bf16_bits(float x) { /* round to nearest even */
  uint32_t u;
  memcpy(&u, &x, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

#define CHECK(cond, ...)                                   \
  do {                                                     \
    if (!(cond)) {                                         \
      fprintf(stderr, "check failed: " __VA_ARGS__);       \
      fprintf(stderr, "\n");                               \
      return 1;                                            \
    }                                                      \
  } while (0)
#define HIP(x) CHECK((x) == hipSuccess, "%s", #x)
#define STEPKV(x)                                                               \
  do {                                                                          \
    int rc_ = (x);                                                              \
    CHECK(rc_ == STEPKV_OK, "%s: %s", #x, stepkv_strerror(rc_));                \
  } while (0)

int main(void) {
  int32_t cu[S + 1] = {0}, cu_steps[S + 1] = {0};
  for (int s = 0; s < S; ++s) {
    cu[s + 1] = cu[s] + kLens[s];
    cu_steps[s + 1] = cu_steps[s] + STEPS;
  }
  const int ntot = cu[S];
  const size_t nq = (size_t)L * S * W * HQ * D, nk = (size_t)L * HKV * ntot * D;
  uint16_t* q = malloc(nq * 2);
  uint16_t* k = malloc(nk * 2);
  uint16_t* v = malloc(nk * 2);
  for (size_t i = 0; i < nq; ++i) q[i] = bf16_bits(2.0f * next_uniform());
  for (size_t i = 0; i < nk; ++i) k[i] = bf16_bits(next_uniform());
  for (size_t i = 0; i < nk; ++i) v[i] = bf16_bits(next_uniform());
  int32_t* sid = malloc(sizeof(int32_t) * ntot);
  uint8_t* prot = malloc(ntot);
  for (int s = 0; s < S; ++s)
    for (int i = 0; i < kLens[s]; ++i) {
      const int n_pr = kLens[s] - PROT;
      prot[cu[s] + i] = i < PROT;
      sid[cu[s] + i] = i < PROT ? -1 : (i - PROT) * STEPS / n_pr;
    }
  float util[S * STEPS];
  for (int j = 0; j < S * STEPS; ++j) util[j] = 0.5f * (float)(j % STEPS) + 0.25f;

  /* device copies */
  void *dq, *dk, *dv, *dsid, *dprot, *dutil, *dcu, *dcus, *dscores, *dsal, *dws, *didx, *dcur;
  HIP(hipMalloc(&dq, nq * 2));
  HIP(hipMalloc(&dk, nk * 2));
  HIP(hipMalloc(&dv, nk * 2));
  HIP(hipMalloc(&dsid, sizeof(int32_t) * ntot));
  HIP(hipMalloc(&dprot, ntot));
  HIP(hipMalloc(&dutil, sizeof util));
  HIP(hipMalloc(&dcu, sizeof cu));
  HIP(hipMalloc(&dcus, sizeof cu_steps));
  HIP(hipMemcpy(dq, q, nq * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dk, k, nk * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dv, v, nk * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dsid, sid, sizeof(int32_t) * ntot, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dprot, prot, ntot, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dutil, util, sizeof util, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dcu, cu, sizeof cu, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dcus, cu_steps, sizeof cu_steps, hipMemcpyHostToDevice));

  void* dstatus;
  HIP(hipMalloc(&dstatus, sizeof(uint32_t)));
  HIP(hipMemset(dstatus, 0, sizeof(uint32_t)));
  stepkv_problem pb = {L, HQ, HKV, D, W, S, cu, dcu, cu_steps, dcus, (uint32_t*)dstatus};
  stepkv_params prm;
  stepkv_params_default(&prm);
  const size_t ws = stepkv_score_workspace_bytes(&pb);
  CHECK(ws > 0, "workspace size");
  const size_t nrow = (size_t)L * HKV * ntot;
  HIP(hipMalloc(&dscores, sizeof(float) * nrow));
  HIP(hipMalloc(&dsal, sizeof(float) * nrow));
  HIP(hipMalloc(&dws, ws));
  STEPKV(stepkv_score(&pb, &prm, dq, dk, dsid, dprot, dutil, dscores, dsal, NULL, dws, ws, NULL));

  int32_t cu_host[S + 1];
  STEPKV(stepkv_retained_rows(&pb, prot, BUDGET, NULL, cu_host));
  const int32_t out_rows = cu_host[S];
  const size_t nout = (size_t)L * HKV * out_rows * D;
  void *dko, *dvo;
  HIP(hipMalloc(&didx, sizeof(int32_t) * nrow));
  HIP(hipMalloc(&dcur, sizeof cu));
  HIP(hipMalloc(&dko, nout * 2));
  HIP(hipMalloc(&dvo, nout * 2));
  STEPKV(stepkv_select(&pb, dscores, dprot, dsid, BUDGET, NULL, didx, dcur, NULL, NULL));
  STEPKV(stepkv_compact(&pb, dk, dv, didx, dcur, out_rows, dko, dvo, NULL));
  /* the same pass as one call, its scores and positions kept in its workspace */
  const size_t cws = stepkv_compress_workspace_bytes(&pb);
  CHECK(cws >= ws, "compress workspace size");
  void *dcws, *dcur2, *dko2, *dvo2;
  HIP(hipMalloc(&dcws, cws));
  HIP(hipMalloc(&dcur2, sizeof cu));
  HIP(hipMalloc(&dko2, nout * 2));
  HIP(hipMalloc(&dvo2, nout * 2));
  STEPKV(stepkv_compress(&pb, &prm, dq, dk, dv, NULL, dsid, dprot, dutil, BUDGET, NULL, NULL, NULL,
                         dcur2, out_rows, dko2, dvo2, dcws, cws, NULL));
  HIP(hipDeviceSynchronize());
  uint32_t flags = 0xffffffffu;
  STEPKV(stepkv_status_read(&pb, &flags, 1, NULL));
  CHECK(flags == 0u, "device status 0x%x on clean inputs", flags);

  float* sal = malloc(sizeof(float) * nrow);
  float* sc = malloc(sizeof(float) * nrow);
  int32_t* idx = malloc(sizeof(int32_t) * nrow);
  int32_t cur[S + 1];
  uint16_t* ko = malloc(nout * 2);
  uint16_t* vo = malloc(nout * 2);
  HIP(hipMemcpy(sal, dsal, sizeof(float) * nrow, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(sc, dscores, sizeof(float) * nrow, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(idx, didx, sizeof(int32_t) * nrow, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(cur, dcur, sizeof cur, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(ko, dko, nout * 2, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(vo, dvo, nout * 2, hipMemcpyDeviceToHost));
  {
    int32_t cur2[S + 1];
    uint16_t* ko2 = malloc(nout * 2);
    uint16_t* vo2 = malloc(nout * 2);
    HIP(hipMemcpy(cur2, dcur2, sizeof cur2, hipMemcpyDeviceToHost));
    HIP(hipMemcpy(ko2, dko2, nout * 2, hipMemcpyDeviceToHost));
    HIP(hipMemcpy(vo2, dvo2, nout * 2, hipMemcpyDeviceToHost));
    CHECK(memcmp(cur2, cur, sizeof cur) == 0 && memcmp(cu_host, cur, sizeof cur) == 0,
          "cu_retained of compress, select and the host rule");
    CHECK(memcmp(ko2, ko, nout * 2) == 0 && memcmp(vo2, vo, nout * 2) == 0,
          "compress equals score, select, compact");
    free(ko2);
    free(vo2);
  }

  const double rows = (double)W * (HQ / HKV);
  CHECK(cur[0] == 0, "cu_retained[0]");
  for (int s = 0; s < S; ++s) {
    const int n_pr = kLens[s] - PROT, keep = PROT + (BUDGET < n_pr ? BUDGET : n_pr);
    CHECK(cur[s + 1] - cur[s] == keep, "retained rows of sequence %d", s);
  }
  for (int lh = 0; lh < L * HKV; ++lh)
    for (int s = 0; s < S; ++s) {
      double mass = 0.0;
      for (int i = 0; i < kLens[s]; ++i) {
        const size_t e = (size_t)lh * ntot + cu[s] + i;
        mass += sal[e];
        if (prot[cu[s] + i]) CHECK(isinf(sc[e]) && sc[e] < 0, "protected score at %zu", e);
        else CHECK(isfinite(sc[e]) && sc[e] >= 0.0f, "prunable score at %zu", e);
      }
      CHECK(fabs(mass - rows) < 1e-3 * rows, "saliency mass %.6f of (head %d, seq %d)", mass, lh, s);
      const int nkeep = cur[s + 1] - cur[s];
      for (int j = 0; j < nkeep; ++j) {
        const int pos = idx[(size_t)lh * ntot + cu[s] + j];
        CHECK(pos >= 0 && pos < kLens[s], "retained position range");
        if (j < PROT) CHECK(pos == j, "protected prefix kept in order");
        if (j > 0) CHECK(pos > idx[(size_t)lh * ntot + cu[s] + j - 1], "ascending positions");
        const size_t src = ((size_t)lh * ntot + cu[s] + pos) * D;
        const size_t dst = ((size_t)lh * out_rows + cur[s] + j) * D;
        CHECK(memcmp(ko + dst, k + src, 2 * D) == 0 && memcmp(vo + dst, v + src, 2 * D) == 0,
              "compacted row (head %d, seq %d, row %d)", lh, s, j);
      }
    }
  printf("ok: %d layers x %d KV heads, %d tokens in %d sequences, %d retained rows\n", L, HKV,
         ntot, S, out_rows);
  return 0;
}
