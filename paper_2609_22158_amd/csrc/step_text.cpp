// Host engine for the step signals of Sec. 5.1 computed from a trajectory's
// text: observation validity, evidence gain and action redundancy (new-step
// scoring, Sec. 5.1.1) and the observation similarities of the reuse update
// (eq. reuse, Sec. 5.1.2), over at most 64 evidence cues per field (App. D).
//
// The paper names an overlap-based similarity of extracted cues without
// fixing either. Here a cue is a maximal run of ASCII letters and digits,
// lowercased, of two or more bytes and not a stop word; a field keeps its
// distinct cues in order of first appearance, the first 64; similarity is
// the Jaccard overlap of two cue sets. Cues are kept as 64-bit FNV-1a hashes
// of their lowercased bytes, so a trajectory's state is a flat array the
// caller owns. Work per boundary is O(t) set comparisons of at most 64 cues.
#include <algorithm>
#include <cstddef>
#include <cstdint>
#include <cstring>

#include "stepkv.h"

namespace {

constexpr uint32_t kMagic = 0x74786b73u;
constexpr int kCap = STEPKV_CUE_CAP;
constexpr int kFields = 3;  // thought followed by observation, action, observation
enum Field { kThObs = 0, kAct = 1, kObs = 2 };

struct StateHeader {
  uint32_t magic;
  int32_t capacity;
  int32_t steps;
  int32_t reserved;
};

// Layout after the header: uint64 cues[capacity][3][64], each field sorted
// ascending, then int32 counts[capacity][3].
size_t cue_offset() { return sizeof(StateHeader); }
size_t count_offset(int capacity) {
  return cue_offset() + sizeof(uint64_t) * (size_t)capacity * kFields * kCap;
}

// Function words that carry no evidence, sorted for binary search.
const char* const kStop[] = {
    "a",      "about", "above",   "again", "all",   "also",  "am",    "an",    "and",   "another",
    "any",    "are",   "as",      "at",    "be",    "been",  "being", "below", "both",  "but",
    "by",     "can",   "could",   "did",   "do",    "does",  "done",  "down",  "each",  "either",
    "for",    "from",  "had",     "has",   "have",  "having", "he",   "her",   "here",  "hers",
    "him",    "his",   "how",     "if",    "in",    "into",  "is",    "it",    "its",   "just",
    "may",    "me",    "might",   "mine",  "more",  "most",  "must",  "my",    "neither", "no",
    "nor",    "not",   "of",      "off",   "on",    "once",  "only",  "onto",  "or",    "other",
    "our",    "ours",  "out",     "over",  "own",   "same",  "shall", "she",   "should", "so",
    "some",   "such",  "than",    "that",  "the",   "their", "theirs", "them", "then",  "there",
    "these",  "they",  "this",    "those", "to",    "too",   "under", "up",    "us",    "very",
    "was",    "we",    "were",    "what",  "when",  "where", "which", "who",   "whom",  "whose",
    "why",    "will",  "with",    "without", "would", "yet", "you",   "your",  "yours",
};
constexpr int kNumStop = sizeof(kStop) / sizeof(kStop[0]);

// Prefixes (after leading ASCII whitespace, case-insensitive) that mark an
// error-returning observation (Sec. 5.1.1 remark).
const char* const kErrorMarkers[] = {"error",      "exception", "traceback", "invalid",
                                     "failed",     "failure",   "no results", "not found",
                                     "timed out",  "timeout"};

inline bool is_alnum(unsigned char c) {
  return (c >= '0' && c <= '9') || (c >= 'a' && c <= 'z') || (c >= 'A' && c <= 'Z');
}
inline unsigned char lower(unsigned char c) { return (c >= 'A' && c <= 'Z') ? c + 32 : c; }
inline bool is_space(unsigned char c) {
  return c == ' ' || c == '\t' || c == '\n' || c == '\r' || c == '\f' || c == '\v';
}

bool is_stop(const unsigned char* p, int64_t n) {
  if (n > 8) return false;  // no stop word is longer
  char w[9];
  for (int64_t i = 0; i < n; ++i) w[i] = (char)lower(p[i]);
  w[n] = '\0';
  int lo = 0, hi = kNumStop - 1;
  while (lo <= hi) {
    const int mid = (lo + hi) / 2;
    const int c = std::strcmp(w, kStop[mid]);
    if (c == 0) return true;
    if (c < 0) hi = mid - 1; else lo = mid + 1;
  }
  return false;
}

uint64_t fnv1a_lower(const unsigned char* p, int64_t n) {
  uint64_t h = 14695981039346656037ull;
  for (int64_t i = 0; i < n; ++i) {
    h ^= lower(p[i]);
    h *= 1099511628211ull;
  }
  return h;
}

// Appends the cues of text[0, n) to out[0, *count), skipping cues already
// there, until the cap. Returns false once the cap is reached.
bool add_cues(const unsigned char* text, int64_t n, uint64_t* out, int* count) {
  int64_t i = 0;
  while (i < n) {
    if (*count == kCap) return false;
    while (i < n && !is_alnum(text[i])) ++i;
    int64_t j = i;
    while (j < n && is_alnum(text[j])) ++j;
    const int64_t len = j - i;
    if (len >= 2 && !is_stop(text + i, len)) {
      const uint64_t h = fnv1a_lower(text + i, len);
      bool seen = false;
      for (int k = 0; k < *count && !seen; ++k) seen = out[k] == h;
      if (!seen) out[(*count)++] = h;
    }
    i = j;
  }
  return *count < kCap;
}

bool starts_with_error_marker(const unsigned char* text, int64_t n) {
  int64_t i = 0;
  while (i < n && is_space(text[i])) ++i;
  for (const char* m : kErrorMarkers) {
    const int64_t len = (int64_t)std::strlen(m);
    if (n - i < len) continue;
    bool eq = true;
    for (int64_t k = 0; k < len && eq; ++k) eq = lower(text[i + k]) == (unsigned char)m[k];
    if (eq) return true;
  }
  return false;
}

// Jaccard overlap of two sorted cue sets (a branch-free merge).
double jaccard(const uint64_t* a, int na, const uint64_t* b, int nb) {
  int i = 0, j = 0, both = 0;
  while (i < na && j < nb) {
    const uint64_t x = a[i], y = b[j];
    both += x == y;
    i += x <= y;
    j += y <= x;
  }
  const int uni = na + nb - both;
  return uni > 0 ? (double)both / (double)uni : 0.0;
}

bool text_ok(const char* p, int64_t n) { return n >= 0 && (n == 0 || p != nullptr); }

}  // namespace

extern "C" {

size_t stepkv_text_state_bytes(int32_t capacity) {
  if (capacity < 1) return 0;
  return count_offset(capacity) + sizeof(int32_t) * (size_t)capacity * kFields;
}

int stepkv_text_state_init(void* state, size_t bytes, int32_t capacity) {
  if (!state || capacity < 1 || bytes < stepkv_text_state_bytes(capacity)) return STEPKV_EINVAL;
  if (reinterpret_cast<uintptr_t>(state) % alignof(uint64_t) != 0) return STEPKV_EINVAL;
  std::memset(state, 0, stepkv_text_state_bytes(capacity));
  StateHeader* h = static_cast<StateHeader*>(state);
  h->magic = kMagic;
  h->capacity = capacity;
  h->steps = 0;
  return STEPKV_OK;
}

int stepkv_text_cues(const char* text, int64_t text_len, uint64_t* cues, int32_t* count) {
  if (!cues || !count || !text_ok(text, text_len)) return STEPKV_EINVAL;
  int n = 0;
  add_cues(reinterpret_cast<const unsigned char*>(text), text_len, cues, &n);
  *count = n;
  return STEPKV_OK;
}

int stepkv_text_step(void* state, const char* thought, int64_t thought_len, const char* action,
                     int64_t action_len, const char* observation, int64_t observation_len,
                     float* valid, float* gain, float* red, float* obs_sim_prev) {
  if (!state || !valid || !gain || !red) return STEPKV_EINVAL;
  if (!text_ok(thought, thought_len) || !text_ok(action, action_len) ||
      !text_ok(observation, observation_len))
    return STEPKV_EINVAL;
  StateHeader* h = static_cast<StateHeader*>(state);
  if (h->magic != kMagic || h->steps < 0 || h->steps >= h->capacity) return STEPKV_EINVAL;
  const int t = h->steps;
  if (t > 0 && !obs_sim_prev) return STEPKV_EINVAL;
  uint8_t* base = static_cast<uint8_t*>(state);
  uint64_t* cues = reinterpret_cast<uint64_t*>(base + cue_offset());
  int32_t* counts = reinterpret_cast<int32_t*>(base + count_offset(h->capacity));
  uint64_t* mine = cues + (size_t)t * kFields * kCap;
  int32_t* my_n = counts + (size_t)t * kFields;

  // the three cue sets of the new step; thought || observation is the thought's
  // cues followed by the observation's (a space separates them)
  const auto* th = reinterpret_cast<const unsigned char*>(thought);
  const auto* ac = reinterpret_cast<const unsigned char*>(action);
  const auto* ob = reinterpret_cast<const unsigned char*>(observation);
  int n_tho = 0, n_act = 0, n_obs = 0;
  if (add_cues(th, thought_len, mine + kThObs * kCap, &n_tho))
    add_cues(ob, observation_len, mine + kThObs * kCap, &n_tho);
  add_cues(ac, action_len, mine + kAct * kCap, &n_act);
  add_cues(ob, observation_len, mine + kObs * kCap, &n_obs);
  *valid = (n_obs > 0 && !starts_with_error_marker(ob, observation_len)) ? 1.0f : 0.0f;
  my_n[kThObs] = n_tho;
  my_n[kAct] = n_act;
  my_n[kObs] = n_obs;
  for (int f = 0; f < kFields; ++f) std::sort(mine + f * kCap, mine + f * kCap + my_n[f]);

  double best_tho = 0.0, best_act = 0.0;
  for (int u = 0; u < t; ++u) {
    const uint64_t* other = cues + (size_t)u * kFields * kCap;
    const int32_t* on = counts + (size_t)u * kFields;
    best_tho = std::max(best_tho, jaccard(mine + kThObs * kCap, n_tho, other + kThObs * kCap,
                                          on[kThObs]));
    best_act = std::max(best_act, jaccard(mine + kAct * kCap, n_act, other + kAct * kCap,
                                          on[kAct]));
    obs_sim_prev[u] =
        (float)jaccard(mine + kObs * kCap, n_obs, other + kObs * kCap, on[kObs]);
  }
  *gain = t == 0 ? 1.0f : (float)(1.0 - best_tho);  // gain_1 = 1
  *red = t == 0 ? 0.0f : (float)best_act;           // red_1 = 0
  h->steps = t + 1;
  return STEPKV_OK;
}

}  // extern "C"
