"""Shared helpers for the GPU parity tests: run the HIP path and the oracle on
the same seeded workload and compare them.

The oracle never receives anything the HIP path produced; the GPU select may
receive the oracle's priorities (cast to fp32) so that both sides rank the
very same numbers.
"""
from __future__ import annotations

import math
import sys

import numpy as np

import oracle as O
from synth import make_workload

SCORE_RTOL = 2e-3  # the stated tolerance for scores from fp32 accumulation of bf16 inputs
ATOL_FRAC = 1e-7   # plus 1e-7 x the per-head max, for values that underflow in fp32


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def oracle_utilities(w) -> np.ndarray:
    out = []
    for sig in w.signals:
        _, _, S = O.run_step_updates(sig.valid, sig.gain, sig.red, sig.obs_sim.astype(np.float64),
                                     O.Params())
        out.append(S)
    return np.concatenate(out) if out else np.zeros(0)


def gpu_utilities(w) -> np.ndarray:
    from paper_2609_22158_amd import binding as B

    out = [B.step_utilities(s.valid, s.gain, s.red, s.obs_sim) for s in w.signals]
    return np.concatenate(out).astype(np.float32) if out else np.zeros(0, np.float32)


def ref_rows(w, budget):
    """The oracle's retained rows per sequence and head."""
    return [O.retained_count(n, p, budget) for n, p in zip(w.seqlens, w.protected_len)]


class HipRun:
    """Device copies of a workload and the HIP path's outputs."""

    def __init__(self, w, budget=None, params=None, want_v=True):
        import torch

        from paper_2609_22158_amd import binding as B

        self.w = w
        self.B = B
        self.budget = w.budget if budget is None else budget
        self.params = params or B.Params()
        self.pb = B.Problem.from_workload(w)
        self.q = B.bf16_from_bits(w.q_win)
        self.k = B.bf16_from_bits(w.k)
        self.v = B.bf16_from_bits(w.v) if want_v and w.v.size else None
        self.sid = torch.from_numpy(w.step_ids).cuda()
        self.prot = torch.from_numpy(w.protected).cuda()
        self.util_host = gpu_utilities(w)
        self.util = torch.from_numpy(self.util_host).cuda()
        self.out_rows = int(self.pb.retained_rows(w.protected, self.budget)[-1])

    def score(self, **kw):
        return self.B.score(self.pb, self.q, self.k, self.sid, self.prot, self.util, self.params,
                            **kw)

    def lse_tensor(self, lse_host: np.ndarray):
        import torch

        return torch.from_numpy(np.ascontiguousarray(lse_host, dtype=np.float32)).cuda()

    def select(self, scores, **kw):
        return self.B.select(self.pb, scores, self.prot, self.sid, self.budget, **kw)

    def compact(self, idx, cu_ret):
        return self.B.compact(self.pb, self.k, self.v, idx, cu_ret, self.out_rows)


def oracle_params(p) -> O.Params:
    return O.Params(alpha=p.alpha, beta=p.beta, pool_kernel=p.pool_kernel,
                    scale=(p.scale if p.scale > 0 else None), causal_tail=bool(p.causal_tail))


def oracle_lse(w, causal: bool, scale=None) -> np.ndarray:
    """Window rows' natural-log log-sum-exp [L][S][W][Hq] from the oracle (fp64)."""
    L, S, W, Hq, d = w.q_win.shape
    G = w.group
    sc = scale if scale is not None else 1.0 / math.sqrt(d)
    out = np.empty((L, S, W, Hq))
    for s in range(S):
        a, b = int(w.cu_seqlens[s]), int(w.cu_seqlens[s + 1])
        for l in range(L):
            qs = O.decode_bf16(w.q_win[l, s])
            for h in range(w.num_kv_heads):
                rows = O.window_rows(qs, h, G)
                keys = O.decode_bf16(w.k[l, h, a:b])
                vis = O.visible_keys(b - a, W, G, causal)
                out[l, s, :, h * G:(h + 1) * G] = O.window_row_lse(rows, keys, sc, vis).reshape(W, G)
    return out


def run_oracle(w, budget, params, heads=None, want_saliency=True, lse_win=None, seqs=None):
    """Oracle results keyed by (s, l, h); `heads` restricts it to some (l, h) pairs and
    `seqs` to some sequences.

    lse_win (natural log, [L][S][W][Hq]) takes the saliency from given row LSEs."""
    S = oracle_utilities(w)
    args = (w.q_win, w.k, None, w.cu_seqlens, w.step_ids, w.protected, w.cu_steps, S, budget,
            oracle_params(params))
    if heads is None:
        res = O.compress(*args, want_saliency=want_saliency, lse_win=lse_win, seqs=seqs)
    else:
        res = None
        for l, h in heads:
            part = O.compress(*args, layers=[l], heads=[h], want_saliency=want_saliency,
                              lse_win=lse_win, seqs=seqs)
            if res is None:
                res = part
            else:
                for name in res:
                    res[name].update(part[name])
    res["S"] = S
    return res


def close(got: np.ndarray, want: np.ndarray, what: str) -> None:
    """|got - want| <= rtol |want| + atol_frac * max|want| elementwise (finite entries)."""
    fin = np.isfinite(want)
    assert np.array_equal(fin, np.isfinite(got)), f"{what}: non-finite pattern differs"
    assert np.array_equal(got[~fin], want[~fin]), f"{what}: infinities differ"
    if not fin.any():
        return
    g, t = got[fin].astype(np.float64), want[fin]
    atol = ATOL_FRAC * float(np.abs(t).max())
    err = np.abs(g - t)
    bad = err > SCORE_RTOL * np.abs(t) + atol
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} outside tolerance; worst "
                           f"rel {float((err / np.maximum(np.abs(t), 1e-300)).max()):.3e}")


def swap_ok(kept_gpu: np.ndarray, kept_oracle: np.ndarray, P: np.ndarray, prunable: np.ndarray,
            budget: int) -> None:
    """Retained prunable sets may differ only by tokens tied with the threshold within tolerance."""
    a = set(int(i) for i in kept_gpu if prunable[i])
    b = set(int(i) for i in kept_oracle if prunable[i])
    assert len(a) == len(b) == min(budget, int(prunable.sum()))
    diff = a ^ b
    if not diff:
        return
    cand = np.sort(P[prunable])[::-1]
    tau = cand[min(budget, cand.size) - 1]
    for i in diff:
        assert abs(P[i] - tau) <= SCORE_RTOL * abs(tau) + 1e-12, (i, P[i], tau)


def reduced(name: str, **kw):
    return make_workload(name, 233, **kw)


def sqrt_d(w) -> float:
    return 1.0 / math.sqrt(w.head_dim)
