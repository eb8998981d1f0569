"""Step signals from a trajectory's text (test infrastructure only).

Paper: "StepKV: Step-Aware KV Cache Compression for LLM Agents", Sec. 5.1.1
(observation validity, evidence gain, action redundancy) and Sec. 5.1.2 (the
reuse update), with the cue cap of the hyper-parameter table (App. D).

The paper calls sim an overlap-based textual similarity over at most 64
extracted evidence cues per field and defines neither a cue nor the overlap.
Readings taken here (the library's host engine implements the same):

* Text is handled as UTF-8 bytes. A cue is a maximal run of ASCII letters and
  digits, lowercased, at least 2 bytes long, and not in STOPWORDS. A field's
  cues are its distinct cues in order of first appearance, the first 64.
* sim(a, b) = |A & B| / |A | B| (Jaccard) over the two cue sets; 0 when both
  are empty.
* An observation is unusable (valid = 0) when it has no cue, or when its
  text, after leading ASCII whitespace and lowercased, starts with one of
  ERROR_MARKERS (an error-returning observation, Sec. 5.1.1 remark).
* gain_k = 1 - max over u < k of sim(cues(Th_k + " " + Obs_k), cues(Th_u + " " + Obs_u));
  gain_1 = 1.
* red_k = max over u < k of sim(cues(Act_k), cues(Act_u)); red_1 = 0.
* The reuse update at boundary t uses sim(cues(Obs_t), cues(Obs_k)) for k < t.
"""
from __future__ import annotations

import re
from typing import List, Sequence, Tuple

import numpy as np

CUE_CAP = 64

# Common English function words: they carry no evidence.
STOPWORDS = frozenset("""
a an the of to in on at by for from with without into onto over under about above below
and or nor but so yet if then than as is are was were be been being am do does did done
has have had having will would can could shall should may might must it its this that
these those there here he she they we you me him her them us his hers their theirs our
ours your yours my mine which who whom whose what when where why how not no also just
only very too more most such some any each all both either neither other another same
own again once up down out off
""".split())

ERROR_MARKERS = ("error", "exception", "traceback", "invalid", "failed", "failure",
                 "no results", "not found", "timed out", "timeout")

_TOKEN = re.compile(rb"[A-Za-z0-9]+")
_WS = b" \t\n\r\f\v"


def _bytes(text) -> bytes:
    return text if isinstance(text, bytes) else str(text).encode("utf-8")


def cues(text) -> List[bytes]:
    """Distinct cues of one field in order of first appearance, at most CUE_CAP."""
    out: List[bytes] = []
    seen = set()
    for m in _TOKEN.finditer(_bytes(text)):
        w = m.group(0).lower()
        if len(w) < 2 or w.decode() in STOPWORDS or w in seen:
            continue
        seen.add(w)
        out.append(w)
        if len(out) == CUE_CAP:
            break
    return out


def sim(a: Sequence[bytes], b: Sequence[bytes]) -> float:
    """Jaccard overlap of two cue sets (0 when both are empty)."""
    A, B = set(a), set(b)
    union = len(A | B)
    return len(A & B) / union if union else 0.0


def observation_valid(obs) -> int:
    """1 when the observation is usable: it has a cue and does not start with an error marker."""
    data = _bytes(obs)
    if not cues(data):
        return 0
    head = data.lstrip(_WS).lower()
    return 0 if any(head.startswith(m.encode()) for m in ERROR_MARKERS) else 1


def step_signals(steps: Sequence[Tuple[str, str, str]]):
    """valid, gain, red [n] and obs_sim [n][n] (obs_sim[t][k] = sim(Obs_t, Obs_k), k < t)
    for a trajectory of (thought, action, observation) steps, in order."""
    n = len(steps)
    valid = np.zeros(n)
    gain = np.zeros(n)
    red = np.zeros(n)
    obs_sim = np.zeros((n, n))
    th_obs, act, obs = [], [], []
    for t, (th, ac, ob) in enumerate(steps):
        th_obs.append(cues(_bytes(th) + b" " + _bytes(ob)))
        act.append(cues(ac))
        obs.append(cues(ob))
        valid[t] = observation_valid(ob)
        gain[t] = 1.0 if t == 0 else 1.0 - max(sim(th_obs[t], th_obs[u]) for u in range(t))
        red[t] = 0.0 if t == 0 else max(sim(act[t], act[u]) for u in range(t))
        for k in range(t):
            obs_sim[t, k] = sim(obs[t], obs[k])
    return valid, gain, red, obs_sim
