"""Shared-index mode (saliency of the last layers, one ranking per sequence, one
retained set for every layer and head), HIP path vs the oracle's compress_shared.

Tolerances as in the per-head parity tests: scores and the summed saliency
within 2e-3 relative (+1e-7 of the sequence's max); selection bit-exact on the
oracle's priorities cast to fp32; compaction bit-exact.
"""
import numpy as np
import pytest

import oracle as O
from paper_2609_22158_amd import binding as B
from tests.gpu_cases import (HipRun, close, log, oracle_lse, oracle_params, oracle_utilities,
                             reduced, swap_ok)

pytestmark = pytest.mark.gpu

CASES = {
    "l4_5003": dict(name="l32_32k", num_layers=4, seqlens=[5003], num_steps=20),  # last 3 of 4
    "ragged_g7": dict(name="ragged16", num_layers=2, seqlens=[2500, 700, 130, 1, 0, 4097],
                      protected_len=64),  # fewer layers than asked for: all of them
    "tiny": dict(name="tiny"),
    # W = 48 at G = 7: 336 window rows per head, two pairs of sweeps
    "ragged_w48": dict(name="ragged16", num_layers=3, window=48, seqlens=[1200, 90, 2222],
                       protected_len=40),
}
LAST = 3

_c = {}


def _case(cid):
    if cid not in _c:
        spec = dict(CASES[cid])
        w = reduced(spec.pop("name"), **spec)
        g = HipRun(w)
        log(f"[shared {cid}] L={w.num_layers} seqlens={w.seqlens} W={w.window} G={w.group}")
        sc = B.score_shared(g.pb, g.q, g.k, g.sid, g.prot, g.util, g.params, last_layers=LAST,
                            want_saliency=True)
        o = _oracle(w, g.budget, g.params)
        _c[cid] = (w, g, sc, o)
    return _c[cid]


def _oracle(w, budget, params, lse_win=None, seqs=None):
    return O.compress_shared(w.q_win, w.k, w.v, w.cu_seqlens, w.step_ids, w.protected, w.cu_steps,
                             oracle_utilities(w), budget, oracle_params(params), last_layers=LAST,
                             lse_win=lse_win, seqs=seqs)


def _seqs(w):
    for s in range(w.num_seqs):
        yield s, int(w.cu_seqlens[s]), int(w.cu_seqlens[s + 1])


@pytest.mark.parametrize("cid", list(CASES))
def test_shared_priority_paths_agree(cid):
    """Without step statistics the priority row of a sequence is spread over many workgroups;
    with them one workgroup per sequence also forms the statistics. Both give the same summed
    saliency and priorities bit for bit, and the statistics count every prunable token once."""
    w, g, sc, o = _case(cid)
    log(f"[shared {cid}] with step statistics")
    sc2 = B.score_shared(g.pb, g.q, g.k, g.sid, g.prot, g.util, g.params, last_layers=LAST,
                         want_saliency=True, want_stats=True)
    assert np.array_equal(sc2["saliency"].cpu().numpy(), sc["saliency"].cpu().numpy())
    assert np.array_equal(sc2["scores"].cpu().numpy(), sc["scores"].cpu().numpy())
    cnt = B.decode_stats(sc2["stats_raw"])["count"].reshape(-1)
    for s, a, b in _seqs(w):
        k0, k1 = int(w.cu_steps[s]), int(w.cu_steps[s + 1])
        prun = w.protected[a:b] == 0
        sid = w.step_ids[a:b]
        want = np.bincount(sid[prun & (sid >= 0) & (sid < k1 - k0)], minlength=k1 - k0)
        assert np.array_equal(cnt[k0:k1], want), f"counts seq {s}"


@pytest.mark.parametrize("pool", [1, 63])
def test_shared_priority_paths_agree_any_pool(pool):
    """The two shared-index priority paths at the smallest and largest pooling windows (a
    halo of 31 positions on each side of a 256-position chunk)."""
    cid = list(CASES)[-1]
    w, g, _, _ = _case(cid)
    p = B.Params(pool_kernel=pool)
    log(f"[shared {cid}] pool {pool}, both priority paths")
    a = B.score_shared(g.pb, g.q, g.k, g.sid, g.prot, g.util, p, last_layers=LAST)
    b = B.score_shared(g.pb, g.q, g.k, g.sid, g.prot, g.util, p, last_layers=LAST,
                       want_stats=True)
    assert np.array_equal(a["scores"].cpu().numpy(), b["scores"].cpu().numpy())


@pytest.mark.parametrize("cid", list(CASES))
def test_shared_scores_match_oracle(cid):
    w, g, sc, o = _case(cid)
    P = sc["scores"].cpu().numpy()
    A = sc["saliency"].cpu().numpy()
    n = min(LAST, w.num_layers)
    for s, a, b in _seqs(w):
        close(A[a:b], o["A"][s], f"A seq {s}")
        close(P[a:b], o["P"][s], f"P seq {s}")
        if b > a:
            mass = n * w.num_kv_heads * w.window * w.group
            assert abs(A[a:b].sum() - mass) < 1e-3 * mass


def _oracle_p32(w, o):
    P = np.full(w.total_tokens, -np.inf, np.float32)
    for s, a, b in _seqs(w):
        P[a:b] = o["P"][s].astype(np.float32)
    return P


@pytest.mark.parametrize("cid", list(CASES))
def test_shared_select_and_compact_bitexact(cid):
    import torch

    w, g, sc, o = _case(cid)
    P32 = _oracle_p32(w, o)
    # the oracle ranks the same fp32 numbers
    o32 = {}
    for s, a, b in _seqs(w):
        prun = w.protected[a:b] == 0
        o32[s] = O.select_retained(P32[a:b].astype(np.float64), prun, g.budget)
    r = B.select_shared(g.pb, torch.from_numpy(P32).cuda(), g.prot, g.sid, g.budget,
                        want_kept=True)
    idx = r["idx"].cpu().numpy()
    cu = r["cu_retained"].cpu().numpy()
    kept = r["kept"].cpu().numpy()
    for s, a, b in _seqs(w):
        R = cu[s + 1] - cu[s]
        assert R == len(o32[s])
        np.testing.assert_array_equal(idx[a:a + R], o32[s])
        k0, k1 = int(w.cu_steps[s]), int(w.cu_steps[s + 1])
        np.testing.assert_array_equal(
            kept[k0:k1], O.kept_per_step(o32[s], w.step_ids[a:b], w.protected[a:b] == 0, k1 - k0))
    out_rows = int(cu[-1])
    k_out, v_out = B.compact_shared(g.pb, g.k, g.v, r["idx"], r["cu_retained"], out_rows)
    ko = k_out.view(torch.int16).cpu().numpy().view(np.uint16)
    vo = v_out.view(torch.int16).cpu().numpy().view(np.uint16)
    for s, a, b in _seqs(w):
        rows = slice(cu[s], cu[s + 1])
        for l in range(w.num_layers):
            for h in range(w.num_kv_heads):
                np.testing.assert_array_equal(ko[l, h, rows], w.k[l, h, a:b][o32[s]])
                np.testing.assert_array_equal(vo[l, h, rows], w.v[l, h, a:b][o32[s]])


@pytest.mark.parametrize("cid", list(CASES))
def test_shared_end_to_end_within_ties(cid):
    w, g, sc, o = _case(cid)
    r = B.select_shared(g.pb, sc["scores"], g.prot, g.sid, g.budget)
    idx = r["idx"].cpu().numpy()
    cu = r["cu_retained"].cpu().numpy()
    for s, a, b in _seqs(w):
        R = cu[s + 1] - cu[s]
        prun = w.protected[a:b] == 0
        swap_ok(idx[a:a + R], o["idx"][s], o["P"][s], prun, g.budget)


def test_shared_per_sequence_ratio_budgets():
    """B_t = max(1, floor(rho N_pr)) per sequence (eq. problem), passed as `budgets`."""
    import torch

    w, g, sc, o = _case("ragged_g7")
    rho = 0.2
    budgets = []
    for s, a, b in _seqs(w):
        budgets.append(O.budget_from_ratio(rho, int((w.protected[a:b] == 0).sum())))
    P32 = _oracle_p32(w, o)
    r = B.select_shared(g.pb, torch.from_numpy(P32).cuda(), g.prot, g.sid, 1,
                        budgets=torch.tensor(budgets, dtype=torch.int32).cuda())
    idx = r["idx"].cpu().numpy()
    cu = r["cu_retained"].cpu().numpy()
    for (s, a, b), bud in zip(_seqs(w), budgets):
        want = O.select_retained(P32[a:b].astype(np.float64), w.protected[a:b] == 0, bud)
        np.testing.assert_array_equal(idx[a:a + cu[s + 1] - cu[s]], want)


@pytest.mark.parametrize("causal", [0, 1])
def test_shared_lse_fed_matches_oracle(causal):
    w, g, _, _ = _case("l4_5003")
    params = B.Params(causal_tail=causal)
    lse32 = oracle_lse(w, bool(causal)).astype(np.float32)
    sc = B.score_shared(g.pb, g.q, g.k, g.sid, g.prot, g.util, params, last_layers=LAST,
                        lse=g.lse_tensor(lse32), want_saliency=True)
    o = _oracle(w, g.budget, params, lse_win=lse32.astype(np.float64))
    P = sc["scores"].cpu().numpy()
    A = sc["saliency"].cpu().numpy()
    for s, a, b in _seqs(w):
        close(A[a:b], o["A"][s], f"lse-fed A seq {s}")
        close(P[a:b], o["P"][s], f"lse-fed P seq {s}")
