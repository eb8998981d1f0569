"""Plain fp64 reference of StepKV's compression pass (test infrastructure only).

Paper: "StepKV: Step-Aware KV Cache Compression for LLM Agents".

Each function restates one definition of the paper in the paper's order and
notation, with no blocking, fusion or streaming beyond what the definition
states; numpy's matmul, exp and stable sort are the only library steps.
Floating point is fp64 throughout, on values decoded exactly from bf16 bits.

Readings taken where the paper is silent (the observation-window saliency is
the reading fixed for this build; the paper calls T_i a conventional
attention-based saliency, Sec. 5.2):

* z[r, i] = scale * q_r . k_i for the window rows r = (w, g), w in [0, W),
  g in [0, G), query head h*G + g; every cached key i of the sequence is
  visible to every window row (no causal mask); scale = 1/sqrt(d).
  With causal_tail, window slot w is instead the query at position
  N - W + w of the sequence and sees keys 0 .. N - W + w only, as in the
  causal attention of the observation prefill that collects T_i (App. C.2);
  a row that sees no key contributes nothing.
* A[i] = sum over rows r of the row-softmax of z (sum, not mean). Given each
  row's log-sum-exp lse_r over its visible keys (which the prefill's
  attention produces), the same A[i] is sum_r exp(z[r, i] - lse_r).
* T = 1-D average pool of A restricted to prunable tokens: window k (odd),
  stride 1, zero padding, divisor k, never crossing the sequence ends;
  protected tokens contribute zero.
* T_hat = T / max over prunable T (0 when that max is 0), so T_hat lies in
  [0, 1] as the score-range analysis assumes (App. C.1).
* P_i = alpha * T_hat_i + beta * S_{s(i)} for prunable i (eq. token-priority).
* Keep the first min(B, N_pr) prunable tokens in a stable order by
  (P descending, position ascending); NaN ranks as -inf and -0.0 as +0.0;
  protected tokens are always kept and not counted in B (eq. problem).
* Retained order is ascending position over protected and kept tokens.
* Shared-index mode (the paper's setting: token saliency from the last 3
  layers, App. D hyper-parameter table; one global ranking of a sequence's
  tokens, Sec. 5.2): A is summed over the last n layers and all their KV
  heads, pooled, normalised and fused once per sequence, and the one
  retained set indexes the cache of every layer and head.
* Step utility follows Algorithm 1, phases 1 and 2, boundary by boundary;
  gain_1 = 1 and red_1 = 0 by definition (Sec. 5.1.1); log is natural.

Parity pins (tests/test_oracle_pins.py): every function below is pinned by
closed forms, library routines it does not use, invariants or hand-derived
values; none is "parity unpinned".
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np

__all__ = [
    "Params",
    "decode_bf16",
    "completion_score",
    "step_utility",
    "run_step_updates",
    "budget_from_ratio",
    "window_rows",
    "visible_keys",
    "window_attention",
    "window_row_lse",
    "window_saliency",
    "window_saliency_from_lse",
    "pooled_saliency",
    "normalised_saliency",
    "priority",
    "select_retained",
    "retained_count",
    "kept_per_step",
    "step_statistics",
    "compact",
    "decode_attention",
    "score_head",
    "compress",
    "compress_shared",
]


@dataclasses.dataclass
class Params:
    """Hyper-parameters; defaults are the paper's (App. D, hyper-parameter table)."""

    alpha: float = 0.2  # token-saliency weight
    beta: float = 0.8  # step-utility weight
    pool_kernel: int = 7
    scale: Optional[float] = None  # None -> 1/sqrt(d)
    lam: float = 0.3  # redundancy penalty lambda
    w_r: float = 0.85
    w_c: float = 0.15
    r_min: float = -1.0
    r_max: float = 2.0
    s_max: float = 8.0
    eta: float = 1.5
    causal_tail: bool = False  # window slot w sees only keys 0 .. N - W + w


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) to float64; every bf16 value is exact in fp64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


# ---------------------------------------------------------------- step utility
def completion_score(valid: float, gain: float, red: float, lam: float) -> float:
    """eq. reward: r_k = valid_k + gain_k - lambda * red_k."""
    return float(valid) + float(gain) - lam * float(red)


def step_utility(r: float, c: float, p: Params) -> float:
    """eq. step-score: S_k = clip(w_r clip(r_k, r_min, r_max) + w_c log(1 + c_k), 0, S_max)."""
    inner = min(max(r, p.r_min), p.r_max)
    val = p.w_r * inner + p.w_c * math.log(1.0 + c)
    return min(max(val, 0.0), p.s_max)


def run_step_updates(valid: Sequence[float], gain: Sequence[float], red: Sequence[float],
                     obs_sim: np.ndarray, p: Params):
    """Algorithm 1, phases 1-2, applied at the boundaries t = 1..n in turn.

    Phase 1 scores the new step t (eq. reward) with c_t = 0 and sets S_t
    (eq. step-score). Phase 2 raises c_k for every earlier step k by
    min(1, eta * sim(Obs_t, Obs_k)) (eq. reuse) and recomputes S_k.
    ``obs_sim[t, k]`` is sim(Obs_t, Obs_k) for k < t (0-based steps).
    Returns (r, c, S) after the last boundary.
    """
    n = len(valid)
    r = [0.0] * n
    c = [0.0] * n
    S = [0.0] * n
    for t in range(n):
        g = 1.0 if t == 0 else float(gain[t])  # gain_1 = 1
        rd = 0.0 if t == 0 else float(red[t])  # red_1 = 0
        r[t] = completion_score(valid[t], g, rd, p.lam)
        c[t] = 0.0
        S[t] = step_utility(r[t], c[t], p)
        for k in range(t):
            c[k] = c[k] + min(1.0, p.eta * float(obs_sim[t, k]))
            S[k] = step_utility(r[k], c[k], p)
    return np.array(r), np.array(c), np.array(S)


def budget_from_ratio(rho: float, n_prunable: int) -> int:
    """eq. problem: B_t = max(1, floor(rho * N_t)); 1e-9 absorbs fp error in rho*N."""
    return max(1, int(math.floor(rho * n_prunable + 1e-9)))


# ------------------------------------------------------------- token saliency
def window_rows(q_win_ls: np.ndarray, h: int, group: int) -> np.ndarray:
    """Window rows of KV head h: row r = w*G + g is query head h*G + g at window slot w.

    q_win_ls: [W][Hq][d] (one layer, one sequence). Returns [W*G][d].
    """
    W, _, d = q_win_ls.shape
    return q_win_ls[:, h * group:(h + 1) * group, :].reshape(W * group, d)


def visible_keys(n_keys: int, window: int, group: int, causal_tail: bool) -> np.ndarray:
    """Boolean [W*G][N]: whether key i is visible to window row r = w*G + g.

    Without causal_tail every key is visible. With it, window slot w is the
    query at position N - W + w and sees keys 0 .. N - W + w (causal prefill).
    """
    rows = window * group
    if not causal_tail:
        return np.ones((rows, n_keys), dtype=bool)
    w = np.arange(rows) // group
    return np.arange(n_keys)[None, :] <= (n_keys - window + w)[:, None]


def _logits(q_rows: np.ndarray, keys: np.ndarray, scale: float,
            visible: Optional[np.ndarray]) -> np.ndarray:
    z = (q_rows @ keys.T) * scale
    return z if visible is None else np.where(visible, z, -np.inf)


def window_attention(q_rows: np.ndarray, keys: np.ndarray, scale: float,
                     visible: Optional[np.ndarray] = None) -> np.ndarray:
    """Row-softmax of z = scale * Q K^T over the visible keys: p[r, i] (fp64).

    Keys a row does not see get 0; a row that sees no key is all 0.
    """
    z = _logits(q_rows, keys, scale, visible)
    m = z.max(axis=1, keepdims=True) if z.shape[1] else np.full((z.shape[0], 1), -np.inf)
    e = np.exp(z - np.where(np.isfinite(m), m, 0.0))
    tot = e.sum(axis=1, keepdims=True)
    return np.divide(e, tot, out=np.zeros_like(e), where=tot > 0)


def window_row_lse(q_rows: np.ndarray, keys: np.ndarray, scale: float,
                   visible: Optional[np.ndarray] = None) -> np.ndarray:
    """Natural-log log-sum-exp of each window row over its visible keys (-inf if none)."""
    z = _logits(q_rows, keys, scale, visible)
    m = z.max(axis=1) if z.shape[1] else np.full(z.shape[0], -np.inf)
    safe = np.where(np.isfinite(m), m, 0.0)
    tot = np.exp(z - safe[:, None]).sum(axis=1)
    with np.errstate(divide="ignore"):
        return np.where(tot > 0, safe + np.log(tot), -np.inf)


def window_saliency(q_rows: np.ndarray, keys: np.ndarray, scale: float,
                    visible: Optional[np.ndarray] = None) -> np.ndarray:
    """A[i] = sum over window rows of the attention row-softmax (sums to the number of
    rows that see at least one key: W*G without a causal tail)."""
    if keys.shape[0] == 0:
        return np.zeros(0)
    return window_attention(q_rows, keys, scale, visible).sum(axis=0)


def window_saliency_from_lse(q_rows: np.ndarray, keys: np.ndarray, scale: float,
                             lse: np.ndarray, visible: Optional[np.ndarray] = None) -> np.ndarray:
    """A[i] = sum over rows r that see key i of exp(z[r, i] - lse_r), given each row's
    log-sum-exp lse_r (natural log) over the keys it sees (App. C.2: T_i comes out of
    the observation prefill, whose attention already normalises every row)."""
    if keys.shape[0] == 0:
        return np.zeros(0)
    z = (q_rows @ keys.T) * scale
    vis = np.ones(z.shape, dtype=bool) if visible is None else visible
    lse = np.asarray(lse, dtype=np.float64)[:, None]
    arg = np.where(vis, z - np.where(np.isfinite(lse), lse, 0.0), -np.inf)
    return np.exp(arg).sum(axis=0)


def pooled_saliency(A: np.ndarray, prunable: np.ndarray, k: int) -> np.ndarray:
    """T[i] = (1/k) * sum of A[j] * prunable[j] over |j - i| <= k // 2, 0 <= j < N."""
    n = A.shape[0]
    half = k // 2
    a = np.where(prunable, A, 0.0)
    T = np.zeros(n)
    for off in range(-half, half + 1):
        lo, hi = max(0, -off), min(n, n - off)
        if lo < hi:
            T[lo:hi] += a[lo + off:hi + off]
    return T / k


def normalised_saliency(T: np.ndarray, prunable: np.ndarray) -> np.ndarray:
    """T_hat = T / max over prunable T, or 0 everywhere when that max is 0."""
    if not prunable.any():
        return np.zeros_like(T)
    m = T[prunable].max()
    if m <= 0.0:
        return np.zeros_like(T)
    return T / m


def priority(T_hat: np.ndarray, step_ids: np.ndarray, S: np.ndarray, prunable: np.ndarray,
             alpha: float, beta: float) -> np.ndarray:
    """eq. token-priority: P_i = alpha T_i + beta S_{s(i)}; protected tokens get -inf.

    A step id outside [0, len(S)) contributes utility 0.
    """
    n = T_hat.shape[0]
    P = np.full(n, -np.inf)
    ok = prunable & (step_ids >= 0) & (step_ids < S.shape[0])
    util = np.zeros(n)
    util[ok] = S[step_ids[ok]]
    P[prunable] = alpha * T_hat[prunable] + beta * util[prunable]
    return P


def select_retained(P: np.ndarray, prunable: np.ndarray, budget: int) -> np.ndarray:
    """Alg. 1 phase 3 and eq. problem: protected tokens plus the top-B prunable.

    Ranking is a stable sort on (P descending, position ascending); NaN ranks
    as -inf, -0.0 as +0.0. Exactly min(B, N_pr) prunable tokens are kept.
    Returns the retained positions in ascending order (int64).
    """
    n = P.shape[0]
    pos = np.arange(n)
    cand = pos[prunable]
    key = np.asarray(P, dtype=np.float64)[prunable].copy()
    key[np.isnan(key)] = -np.inf
    key[key == 0.0] = 0.0  # -0.0 -> +0.0
    order = np.lexsort((cand, -key))
    take = cand[order[:min(int(budget), cand.shape[0])]]
    keep = np.zeros(n, dtype=bool)
    keep[~prunable] = True
    keep[take] = True
    return pos[keep]


def retained_count(n_tokens: int, n_protected: int, budget: int) -> int:
    """eq. problem with the Algorithm 1 output size: every protected token plus
    min(B, N_pr) prunable ones, R = P + min(B, N - P)."""
    return int(n_protected) + min(int(budget), int(n_tokens) - int(n_protected))


def kept_per_step(idx: np.ndarray, step_ids: np.ndarray, prunable: np.ndarray,
                  n_steps: int) -> np.ndarray:
    """Number of retained prunable tokens of every step (a per-step histogram)."""
    out = np.zeros(n_steps, dtype=np.int64)
    for i in idx:
        if prunable[i] and 0 <= step_ids[i] < n_steps:
            out[step_ids[i]] += 1
    return out


def step_statistics(T_hat: np.ndarray, step_ids: np.ndarray, prunable: np.ndarray,
                    n_steps: int) -> Dict[str, np.ndarray]:
    """Per-step token count, max and sum of T_hat over the step's prunable tokens."""
    cnt = np.zeros(n_steps, dtype=np.int64)
    mx = np.zeros(n_steps)
    sm = np.zeros(n_steps)
    for i in range(T_hat.shape[0]):
        k = step_ids[i]
        if prunable[i] and 0 <= k < n_steps:
            cnt[k] += 1
            mx[k] = max(mx[k], T_hat[i])
            sm[k] += T_hat[i]
    return {"count": cnt, "max": mx, "sum": sm}


def compact(K: np.ndarray, V: np.ndarray, idx: np.ndarray):
    """eq. problem: C_hat = C_prot || C_traj[K], as rows gathered in position order."""
    return K[idx], V[idx]


def decode_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float) -> np.ndarray:
    """One decode query against a (compacted) cache: softmax(scale q K^T) V."""
    z = (K @ q) * scale
    e = np.exp(z - z.max())
    return (e / e.sum()) @ V


# ------------------------------------------------------------- whole pass
def score_head(q_rows: np.ndarray, keys: np.ndarray, step_ids: np.ndarray,
               prunable: np.ndarray, S: np.ndarray, p: Params, scale: float,
               window: Optional[int] = None, lse: Optional[np.ndarray] = None):
    """Saliency, pooling, normalisation and priority for one (sequence, layer, KV head).

    window (W) is needed with p.causal_tail; lse (per window row, natural log)
    selects the saliency from given log-sum-exps."""
    visible = None
    if p.causal_tail:
        visible = visible_keys(keys.shape[0], window, q_rows.shape[0] // window, True)
    if lse is None:
        A = window_saliency(q_rows, keys, scale, visible)
    else:
        A = window_saliency_from_lse(q_rows, keys, scale, lse, visible)
    T = pooled_saliency(A, prunable, p.pool_kernel)
    T_hat = normalised_saliency(T, prunable)
    P = priority(T_hat, step_ids, S, prunable, p.alpha, p.beta)
    return A, T_hat, P


def compress(q_win: np.ndarray, k: np.ndarray, v: Optional[np.ndarray], cu_seqlens: np.ndarray,
             step_ids: np.ndarray, protected: np.ndarray, cu_steps: np.ndarray,
             S: np.ndarray, budget: int, p: Params = Params(),
             layers: Optional[Sequence[int]] = None, heads: Optional[Sequence[int]] = None,
             seqs: Optional[Sequence[int]] = None, want_saliency: bool = False,
             lse_win: Optional[np.ndarray] = None) -> Dict:
    """Run the pass over the chosen (sequence, layer, KV head) triples, one at a time.

    Arguments use the library's layouts with bf16 as uint16 bits:
    q_win [L][S][W][Hq][d], k/v [L][Hkv][Ntot][d], step_ids/protected [Ntot],
    S [cu_steps[-1]] (fp64 step utilities), and optionally lse_win [L][S][W][Hq],
    the window rows' natural-log log-sum-exps to take the saliency from.
    Results are keyed by (s, l, h).
    """
    L, nseq, W, Hq, d = q_win.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    scale = p.scale if p.scale is not None else 1.0 / math.sqrt(d)
    out: Dict = {"P": {}, "idx": {}, "T_hat": {}, "A": {}, "k_hat": {}, "v_hat": {},
                 "kept": {}}
    for s in (range(nseq) if seqs is None else seqs):
        a, b = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
        sid = step_ids[a:b]
        prun = protected[a:b] == 0
        Ss = np.asarray(S[int(cu_steps[s]):int(cu_steps[s + 1])], dtype=np.float64)
        for l in (range(L) if layers is None else layers):
            qs = decode_bf16(q_win[l, s])
            for h in (range(Hkv) if heads is None else heads):
                keys = decode_bf16(k[l, h, a:b])
                lse = None
                if lse_win is not None:
                    lse = np.asarray(lse_win[l, s][:, h * G:(h + 1) * G],
                                     dtype=np.float64).reshape(W * G)
                A, T_hat, P = score_head(window_rows(qs, h, G), keys, sid, prun, Ss, p, scale,
                                         window=W, lse=lse)
                idx = select_retained(P, prun, budget)
                key = (s, l, h)
                out["P"][key] = P
                out["idx"][key] = idx
                out["kept"][key] = kept_per_step(idx, sid, prun, Ss.shape[0])
                if want_saliency:
                    out["A"][key] = A
                    out["T_hat"][key] = T_hat
                if v is not None and v.size:
                    out["k_hat"][key] = k[l, h, a:b][idx]
                    out["v_hat"][key] = v[l, h, a:b][idx]
    return out


def compress_shared(q_win: np.ndarray, k: np.ndarray, v: Optional[np.ndarray],
                    cu_seqlens: np.ndarray, step_ids: np.ndarray, protected: np.ndarray,
                    cu_steps: np.ndarray, S: np.ndarray, budget: int, p: Params = Params(),
                    last_layers: int = 3, seqs: Optional[Sequence[int]] = None,
                    lse_win: Optional[np.ndarray] = None, want_kv: bool = True) -> Dict:
    """Shared-index mode: one ranking per sequence from the last `last_layers` layers.

    For sequence s: A[i] = sum over layers l >= L - last_layers and KV heads h of
    that head's window saliency; T, T_hat and P follow from A as in the per-head
    mode; one retained set K_s; the compacted cache of every (l, h) is K[l][h][K_s]
    and V[l][h][K_s]. Results are keyed by s; k_hat / v_hat are [L][Hkv][R_s][d].
    """
    L, nseq, W, Hq, d = q_win.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    n = min(max(int(last_layers), 1), L)
    scale = p.scale if p.scale is not None else 1.0 / math.sqrt(d)
    out: Dict = {"P": {}, "idx": {}, "T_hat": {}, "A": {}, "k_hat": {}, "v_hat": {},
                 "kept": {}}
    for s in (range(nseq) if seqs is None else seqs):
        a, b = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
        sid = step_ids[a:b]
        prun = protected[a:b] == 0
        Ss = np.asarray(S[int(cu_steps[s]):int(cu_steps[s + 1])], dtype=np.float64)
        visible = visible_keys(b - a, W, G, True) if p.causal_tail else None
        A = np.zeros(b - a)
        for l in range(L - n, L):
            qs = decode_bf16(q_win[l, s])
            for h in range(Hkv):
                rows = window_rows(qs, h, G)
                keys = decode_bf16(k[l, h, a:b])
                if lse_win is None:
                    A = A + window_saliency(rows, keys, scale, visible)
                else:
                    lse = np.asarray(lse_win[l, s][:, h * G:(h + 1) * G],
                                     dtype=np.float64).reshape(W * G)
                    A = A + window_saliency_from_lse(rows, keys, scale, lse, visible)
        T = pooled_saliency(A, prun, p.pool_kernel)
        T_hat = normalised_saliency(T, prun)
        P = priority(T_hat, sid, Ss, prun, p.alpha, p.beta)
        idx = select_retained(P, prun, budget)
        out["A"][s] = A
        out["T_hat"][s] = T_hat
        out["P"][s] = P
        out["idx"][s] = idx
        out["kept"][s] = kept_per_step(idx, sid, prun, Ss.shape[0])
        if want_kv:
            out["k_hat"][s] = k[:, :, a:b][:, :, idx]
            if v is not None and v.size:
                out["v_hat"][s] = v[:, :, a:b][:, :, idx]
    return out
