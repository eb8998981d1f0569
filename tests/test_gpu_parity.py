"""HIP path vs the CPU oracle, through the C ABI, on seeded synthetic caches.

Scores and saliency: within 2e-3 relative (+1e-7 of the head's max).
Selection: bit-exact when both sides rank the oracle's priorities cast to
fp32; end to end, retained sets may differ only by tokens whose priority is
tied with the threshold within that tolerance. Compaction: bit-exact.
"""
import numpy as np
import pytest

import oracle as O
from tests.gpu_cases import (HipRun, close, log, oracle_params, reduced, ref_rows, run_oracle,
                              swap_ok)

pytestmark = pytest.mark.gpu

# sizes the oracle finishes in seconds, each spanning several key tiles and a
# ragged tail, covering every window-row shape: W*G = 64, 128, 256, 224, and 448
# (two groups of window rows)
CASES = {
    "tiny": dict(name="tiny"),  # the 1-layer, N=1024, d=64 configuration, unchanged
    "l1_8k": dict(name="l1_8k"),  # the 8B-shaped single layer, N=8192, unchanged
    "l1_tail3001": dict(name="l1_8k", seqlens=[3001]),
    "l32_32k_2l": dict(name="l32_32k", num_layers=2, seqlens=[5003], num_steps=20),
    "ragged_g7": dict(name="ragged16", num_layers=2, seqlens=[2500, 700, 130, 1, 0, 4097],
                      protected_len=64),
    # W = 64 at G = 7: 448 window rows, two pairs of sweeps (256 and 192 rows)
    "ragged_w64": dict(name="ragged16", num_layers=2, window=64, seqlens=[1500, 333, 0, 2100],
                       protected_len=64),
    # 32 sequences (the most whose chunk table the sweeps take as launch
    # arguments) and 40 (found from cu_seqlens in device memory), with empty,
    # one-token and multi-chunk sequences
    "seqs32": dict(name="ragged16", num_layers=1, seqlens=[(53 * i + 7) % 600 for i in range(31)]
                   + [4500], protected_len=64),
    "seqs40": dict(name="ragged16", num_layers=1, seqlens=[(37 * i * i + 11 * i) % 700
                                                           for i in range(39)] + [4500],
                   protected_len=64),
}

_cache = {}


def _case(cid):
    if cid not in _cache:
        spec = dict(CASES[cid])
        name = spec.pop("name")
        log(f"[case {cid}] generating")
        w = reduced(name, **spec)
        g = HipRun(w)
        log(f"[case {cid}] gpu score, L={w.num_layers} seqlens={w.seqlens} W={w.window} "
            f"G={w.group} d={w.head_dim}")
        sc = g.score(want_saliency=True, want_stats=True)
        import torch

        torch.cuda.synchronize()
        log(f"[case {cid}] oracle")
        o = run_oracle(w, g.budget, g.params)
        _cache[cid] = (w, g, sc, o)
    return _cache[cid]


def _heads(w):
    for s in range(w.num_seqs):
        a, b = int(w.cu_seqlens[s]), int(w.cu_seqlens[s + 1])
        for l in range(w.num_layers):
            for h in range(w.num_kv_heads):
                yield s, l, h, a, b


@pytest.mark.parametrize("cid", list(CASES))
def test_scores_and_saliency_match_oracle(cid):
    w, g, sc, o = _case(cid)
    P = sc["scores"].cpu().numpy()
    A = sc["saliency"].cpu().numpy()
    for s, l, h, a, b in _heads(w):
        close(P[l, h, a:b], o["P"][(s, l, h)], f"P{(s, l, h)}")
        close(A[l, h, a:b], o["A"][(s, l, h)], f"A{(s, l, h)}")
        if b > a:
            assert abs(A[l, h, a:b].sum() - w.window * w.group) < 1e-3 * w.window * w.group


@pytest.mark.parametrize("schedule,causal", [(1, 0), (2, 0), (2, 1)])
@pytest.mark.parametrize("cid", ["tiny", "l32_32k_2l", "ragged_g7", "ragged_w64", "seqs40"])
def test_both_sweep_schedules_match_oracle(cid, schedule, causal):
    """One launch per sweep (1) and both sweeps in one launch (2, also with the
    causal tail), whichever the problem would get by itself: saliency and scores
    against the oracle, and the one-launch path reports no stopped wait
    (STEPKV_FLAG_SYNC)."""
    from paper_2609_22158_amd import binding as B

    w, _, _, o = _case(cid)
    g = HipRun(w, params=B.Params(saliency_schedule=schedule, causal_tail=causal))
    if causal:
        o = run_oracle(w, g.budget, g.params)
    log(f"[schedule {schedule} causal {causal} {cid}]")
    g.pb.status(clear=True)
    sc = g.score(want_saliency=True)
    P = sc["scores"].cpu().numpy()
    A = sc["saliency"].cpu().numpy()
    assert g.pb.status(clear=True) == 0
    for s, l, h, a, b in _heads(w):
        close(P[l, h, a:b], o["P"][(s, l, h)], f"P{(s, l, h)} schedule {schedule}")
        close(A[l, h, a:b], o["A"][(s, l, h)], f"A{(s, l, h)} schedule {schedule}")


def test_saliency_with_logit_spikes_matches_oracle():
    """Keys planted late in a key chunk lift one window row's logit by about
    40 and 90 nats above the rest of the row: the first exceeds fp32 exp range
    relative to the chunk's first tile, so the row's running reference has to
    move; the second stays in range and leaves a large running sum."""
    from synth.workloads import bf16_bits_to_f32, f32_to_bf16_bits

    w = reduced("l1_8k", seqlens=[5000])
    q = bf16_bits_to_f32(w.q_win)  # [L][S][W][Hq][d]
    k = w.k.copy()
    G = w.group
    plants = []  # (kv head, key, window row, factor)
    for h in range(w.num_kv_heads):
        for n, (key, factor) in enumerate([(1000, 8.0), (2100, 3.5), (4500, 8.0), (4999, 8.0)]):
            wr, g = (7 * h + 5 * n) % w.window, (h + n) % G
            k[0, h, key] = f32_to_bf16_bits(factor * q[0, 0, wr, h * G + g])
            plants.append((h, key, wr * G + g, factor))
    w.k = k
    g = HipRun(w)
    sc = g.score(want_saliency=True)
    import torch

    torch.cuda.synchronize()
    o = run_oracle(w, g.budget, g.params)
    A = sc["saliency"].cpu().numpy()
    P = sc["scores"].cpu().numpy()
    for h in range(w.num_kv_heads):
        close(A[0, h], o["A"][(0, 0, h)], f"A(0,0,{h}) with spikes")
        close(P[0, h], o["P"][(0, 0, h)], f"P(0,0,{h}) with spikes")
    for h, key, row, factor in plants:  # each spike takes almost all of its row's mass
        assert o["A"][(0, 0, h)][key] > 0.99, (h, key, row, factor)


@pytest.mark.parametrize("cid", list(CASES))
def test_step_statistics_match_oracle(cid):
    from paper_2609_22158_amd import binding as B

    w, g, sc, o = _case(cid)
    st = B.decode_stats(sc["stats_raw"])
    for s, l, h, a, b in _heads(w):
        k0, k1 = int(w.cu_steps[s]), int(w.cu_steps[s + 1])
        prun = w.protected[a:b] == 0
        ref = O.step_statistics(o["T_hat"][(s, l, h)], w.step_ids[a:b], prun, k1 - k0)
        assert np.array_equal(st["count"][l, h, k0:k1], ref["count"])
        np.testing.assert_allclose(st["max"][l, h, k0:k1], ref["max"], rtol=2e-3, atol=1e-6)
        np.testing.assert_allclose(st["sum"][l, h, k0:k1], ref["sum"], rtol=2e-3, atol=1e-4)


def _oracle_scores_fp32(w, o):
    import torch

    P = np.full((w.num_layers, w.num_kv_heads, w.total_tokens), -np.inf, np.float32)
    for s, l, h, a, b in _heads(w):
        P[l, h, a:b] = o["P"][(s, l, h)].astype(np.float32)
    return P, torch.from_numpy(P).cuda()


def _check_selection(w, g, P32, idx, cu_ret, kept, heads=None):
    """GPU selection on the oracle's fp32 priorities == oracle selection on the same numbers."""
    rows = ref_rows(w, g.budget)
    assert list(cu_ret) == list(np.concatenate([[0], np.cumsum(rows)]))
    for s, l, h, a, b in _heads(w):
        if heads is not None and (l, h) not in heads:
            continue
        prun = w.protected[a:b] == 0
        ref = O.select_retained(P32[l, h, a:b], prun, g.budget)
        got = idx[l, h, a:a + rows[s]]
        assert np.array_equal(got, ref), f"idx{(s, l, h)}"
        if kept is not None:
            k0, k1 = int(w.cu_steps[s]), int(w.cu_steps[s + 1])
            ref_k = O.kept_per_step(ref, w.step_ids[a:b], prun, k1 - k0)
            assert np.array_equal(kept[l, h, k0:k1], ref_k), f"kept{(s, l, h)}"


@pytest.mark.parametrize("cid", list(CASES))
def test_select_and_compact_bitexact_on_oracle_scores(cid):
    import torch

    w, g, sc, o = _case(cid)
    P32, Pdev = _oracle_scores_fp32(w, o)
    log(f"[case {cid}] gpu select on oracle priorities")
    idx, cu_ret, kept = g.select(Pdev, want_kept=True)
    k_hat, v_hat = g.compact(idx, cu_ret)
    torch.cuda.synchronize()
    idx, cu_ret, kept = idx.cpu().numpy(), cu_ret.cpu().numpy(), kept.cpu().numpy()
    _check_selection(w, g, P32, idx, cu_ret, kept)
    kh = k_hat.view(torch.int16).cpu().numpy().view(np.uint16)
    vh = v_hat.view(torch.int16).cpu().numpy().view(np.uint16)
    rows = ref_rows(w, g.budget)
    for s, l, h, a, b in _heads(w):
        r0 = int(cu_ret[s])
        sel = idx[l, h, a:a + rows[s]]
        kr, vr = O.compact(w.k[l, h, a:b], w.v[l, h, a:b], sel)
        assert np.array_equal(kh[l, h, r0:r0 + rows[s]], kr), f"k_hat{(s, l, h)}"
        assert np.array_equal(vh[l, h, r0:r0 + rows[s]], vr), f"v_hat{(s, l, h)}"


@pytest.mark.parametrize("cid", list(CASES))
def test_end_to_end_selection_within_ties(cid):
    w, g, sc, o = _case(cid)
    log(f"[case {cid}] gpu select on gpu priorities")
    idx, cu_ret, _ = g.select(sc["scores"])
    idx = idx.cpu().numpy()
    rows = ref_rows(w, g.budget)
    for s, l, h, a, b in _heads(w):
        got = idx[l, h, a:a + rows[s]]
        assert (np.diff(got) > 0).all()
        prun = w.protected[a:b] == 0
        assert set(np.nonzero(~prun)[0]) <= set(got)
        swap_ok(got, o["idx"][(s, l, h)], o["P"][(s, l, h)], prun, g.budget)


@pytest.mark.parametrize("budget", [1, 7, 959, 960, 5000])
def test_budget_edges(budget):
    """B = 1, B one below and at N_pr = 960 (all kept), and B far above N_pr."""
    import torch

    w = reduced("tiny")
    g = HipRun(w, budget=budget)
    log(f"[budget {budget}] gpu")
    sc = g.score()
    idx, cu_ret, kept = g.select(sc["scores"], want_kept=True)
    torch.cuda.synchronize()
    o = run_oracle(w, budget, g.params, want_saliency=False)
    P32, Pdev = _oracle_scores_fp32(w, o)
    idx2, cu2, kept2 = g.select(Pdev, want_kept=True)
    _check_selection(w, g, P32, idx2.cpu().numpy(), cu2.cpu().numpy(), kept2.cpu().numpy())
    n_keep = 64 + min(budget, 960)
    assert int(cu_ret.cpu()[1]) == n_keep
    idx = idx.cpu().numpy()
    for s, l, h, a, b in _heads(w):
        swap_ok(idx[l, h, :n_keep], o["idx"][(s, l, h)], o["P"][(s, l, h)],
                w.protected == 0, budget)


@pytest.mark.parametrize("alpha,beta", [(0.0, 0.8), (0.2, 0.0)])
def test_single_signal_special_cases(alpha, beta):
    """alpha = 0: whole steps by utility; beta = 0: pure pooled-saliency top-B (Table 3 ablations)."""
    from paper_2609_22158_amd import binding as B

    w = reduced("l1_8k", seqlens=[2049])
    p = B.Params(alpha=alpha, beta=beta)
    g = HipRun(w, params=p)
    log(f"[alpha {alpha} beta {beta}] gpu")
    sc = g.score()
    idx, _, _ = g.select(sc["scores"])
    o = run_oracle(w, g.budget, p, want_saliency=False)
    P = sc["scores"].cpu().numpy()
    idx = idx.cpu().numpy()
    rows = ref_rows(w, g.budget)
    for s, l, h, a, b in _heads(w):
        close(P[l, h, a:b], o["P"][(s, l, h)], f"P{(s, l, h)}")
        prun = w.protected[a:b] == 0
        swap_ok(idx[l, h, :rows[0]], o["idx"][(s, l, h)], o["P"][(s, l, h)], prun, g.budget)


@pytest.mark.parametrize("selector", ["token_only", "last_query_only"])
def test_token_only_selectors(selector):
    """Token-only selectors on the same kernels (beta = 0): SnapKV-style (window saliency,
    pooled) and TOVA-style (one window query, no pooling), against the oracle, with the
    selection bit-exact on the oracle's fp32 priorities."""
    import torch

    from paper_2609_22158_amd import binding as B

    w = reduced("l1_8k", seqlens=[3001, 700], window=1 if selector == "last_query_only" else 32)
    p = getattr(B.Params, selector)()
    g = HipRun(w, params=p)
    log(f"[{selector}] W={w.window} pool={p.pool_kernel}")
    sc = g.score(want_saliency=True)
    o = run_oracle(w, g.budget, p)
    P = sc["scores"].cpu().numpy()
    A = sc["saliency"].cpu().numpy()
    for s, l, h, a, b in _heads(w):
        close(A[l, h, a:b], o["A"][(s, l, h)], f"A{(s, l, h)}")
        close(P[l, h, a:b], o["P"][(s, l, h)], f"P{(s, l, h)}")
    P32, Pdev = _oracle_scores_fp32(w, o)
    idx, cu, _ = g.select(Pdev)
    _check_selection(w, g, P32, idx.cpu().numpy(), cu.cpu().numpy(), None)


@pytest.mark.parametrize("pool", [7, 15])
def test_long_sequence_and_wide_pool_match_oracle(pool):
    """A 40000-token sequence (past the 32768 the register paths hold) and a pooling window of
    15 (past the 9 of the batched priority kernel) take the streamed priority kernel; scores,
    saliency and step statistics against the oracle."""
    from paper_2609_22158_amd import binding as B

    w = reduced("ragged16", num_layers=1, seqlens=[40000, 333], protected_len=64, num_steps=30)
    p = B.Params(pool_kernel=pool)
    g = HipRun(w, params=p, want_v=False)
    log(f"[long sequence pool {pool}] gpu score")
    sc = g.score(want_saliency=True, want_stats=True)
    o = run_oracle(w, g.budget, p)
    P = sc["scores"].cpu().numpy()
    A = sc["saliency"].cpu().numpy()
    st = B.decode_stats(sc["stats_raw"])
    for s, l, h, a, b in _heads(w):
        close(A[l, h, a:b], o["A"][(s, l, h)], f"A{(s, l, h)}")
        close(P[l, h, a:b], o["P"][(s, l, h)], f"P{(s, l, h)}")
        k0, k1 = int(w.cu_steps[s]), int(w.cu_steps[s + 1])
        prun = w.protected[a:b] == 0
        ref = O.step_statistics(o["T_hat"][(s, l, h)], w.step_ids[a:b], prun, k1 - k0)
        assert np.array_equal(st["count"][l, h, k0:k1], ref["count"])
        np.testing.assert_allclose(st["max"][l, h, k0:k1], ref["max"], rtol=2e-3, atol=1e-6)
        np.testing.assert_allclose(st["sum"][l, h, k0:k1], ref["sum"], rtol=2e-3, atol=1e-4)


def _special_scores(w, seed):
    """Priorities that stress the key mapping and the radix search, one pattern per
    (layer, KV head): NaNs of both signs (quiet and signalling), signed zeros,
    infinities, subnormals, huge and negative values, all-equal rows, and
    quantised values with many exact ties."""
    rng = np.random.default_rng(seed)
    bits = lambda *u: np.array(u, np.uint32).view(np.float32)
    nans = bits(0x7FC00000, 0xFFC00000, 0x7F800001, 0xFFBFFFFF)
    specials = np.concatenate([nans, np.array(
        [0.0, -0.0, np.inf, -np.inf, 1e-40, -1e-40, 1.4e-45, -1.4e-45, 3e38, -3e38, 0.5, -2.0],
        np.float32)])
    n = w.total_tokens
    pats = [
        lambda: np.where(rng.random(n) < 0.3, rng.choice(specials, n),
                         np.round(rng.random(n) * 16) / 8).astype(np.float32),
        lambda: np.full(n, 0.25, np.float32),                        # every candidate ties
        lambda: (-np.round(rng.random(n) * 64) / 16 - 1).astype(np.float32),  # negative only
        lambda: rng.choice(np.array([np.inf, 3e38, 2e38, 1.7014118e38], np.float32), n),
        lambda: rng.choice(nans, n),                                  # all rank as -inf
        lambda: rng.random(n).astype(np.float32),
        lambda: (rng.integers(-5, 6, n) * np.float32(1.4e-45)).astype(np.float32),  # subnormal
        lambda: rng.choice(specials, n),
    ]
    P = np.empty((w.num_layers, w.num_kv_heads, n), np.float32)
    for lh in range(w.num_layers * w.num_kv_heads):
        P[lh // w.num_kv_heads, lh % w.num_kv_heads] = pats[lh % len(pats)]()
    return P


@pytest.mark.parametrize("seqlens", [[2500, 700, 130, 1, 0, 4097, 32768], [40000, 3001]],
                         ids=["registers", "streamed"])
@pytest.mark.parametrize("budget", [1, 37, 1000, 1024, 1025, 1500, 2048, 2049, 3000, 4096])
def test_select_special_values_bitexact(seqlens, budget):
    """Selection on crafted fp32 priorities == the oracle's stable ranking of the same numbers
    (NaN as -inf, -0 as +0), including the kept-per-step counts; sequences up to 32768 tokens
    take the register path, longer ones the streamed path. The register path bounds tau from
    below by the smallest per-thread m-th largest key: m = 1 for budgets up to the 1024
    threads (1, 37, 1000, 1024), 2 up to 2048 (1025, 1500, 2048) and 4 above (2049, 3000,
    4096); where the bound does not hold for a row it takes the full key range."""
    import torch

    w = reduced("ragged16", num_layers=2, seqlens=seqlens, protected_len=64, with_v=False)
    g = HipRun(w, budget=budget, want_v=False)
    P = _special_scores(w, 7 + budget)
    log(f"[special values {seqlens} B={budget}] gpu select")
    idx, cu_ret, kept = g.select(torch.from_numpy(P).cuda(), want_kept=True)
    torch.cuda.synchronize()
    with np.errstate(invalid="ignore"):  # signalling NaNs quieted by the fp64 cast
        _check_selection(w, g, P, idx.cpu().numpy(), cu_ret.cpu().numpy(), kept.cpu().numpy())


def test_repeat_runs_are_bitwise_identical():
    """Fixed reduction orders: repeated runs give identical bits (idx only where defined)."""
    import torch

    w = reduced("ragged16", num_layers=2, seqlens=[5003, 2100], num_steps=20)
    g = HipRun(w)
    rows = ref_rows(w, g.budget)
    outs = []
    for rep in range(3):
        log(f"[determinism] run {rep}")
        sc = g.score(want_saliency=True, want_stats=True)
        idx, cu, kept = g.select(sc["scores"], want_kept=True)
        k_hat, v_hat = g.compact(idx, cu)
        torch.cuda.synchronize()
        idx = idx.cpu().numpy()
        defined = [idx[:, :, int(w.cu_seqlens[s]):int(w.cu_seqlens[s]) + rows[s]]
                   for s in range(w.num_seqs)]
        outs.append({"scores": sc["scores"].cpu().numpy(),
                     "saliency": sc["saliency"].cpu().numpy(),
                     "stats": sc["stats_raw"].cpu().numpy(), "kept": kept.cpu().numpy(),
                     "idx": np.concatenate(defined, axis=2),
                     "k_hat": k_hat.view(torch.int16).cpu().numpy(),
                     "v_hat": v_hat.view(torch.int16).cpu().numpy()})
    for rep in (1, 2):
        for name, ref in outs[0].items():
            assert np.array_equal(outs[rep][name].view(np.uint8), ref.view(np.uint8)), \
                f"{name} differs in run {rep}"


def test_decode_over_compacted_cache():
    """One decode step over the compacted ragged cache matches textbook attention."""
    import torch

    from paper_2609_22158_amd import binding as B

    w = reduced("ragged16", num_layers=2, seqlens=[2500, 700, 130, 1, 4097], protected_len=64)
    g = HipRun(w)
    o = run_oracle(w, g.budget, g.params, want_saliency=False)
    P32, Pdev = _oracle_scores_fp32(w, o)
    idx, cu_ret, _ = g.select(Pdev)
    k_hat, v_hat = g.compact(idx, cu_ret)
    qd = B.bf16_from_bits(w.q_dec)
    log("[decode] gpu")
    out = B.decode_attention(g.pb, qd, k_hat, v_hat, cu_ret, g.out_rows).cpu().numpy()
    scale = 1.0 / np.sqrt(w.head_dim)
    for s in range(w.num_seqs):
        a, b = int(w.cu_seqlens[s]), int(w.cu_seqlens[s + 1])
        for l in range(w.num_layers):
            for hq in range(w.num_q_heads):
                h = hq // w.group
                sel = o["idx"][(s, l, h)]
                kr, vr = O.compact(w.k[l, h, a:b], w.v[l, h, a:b], sel)
                ref = O.decode_attention(O.decode_bf16(w.q_dec[l, s, hq]), O.decode_bf16(kr),
                                         O.decode_bf16(vr), scale)
                err = np.abs(out[l, s, hq] - ref).max()
                assert err <= 2e-3 * np.abs(ref).max() + 1e-6, (s, l, hq, err)


def test_full_size_lse_fed_configuration_sampled():
    """The bench's --lse-fed configuration at full size (32 layers, 32k tokens, W=64):
    the row LSEs come from stepkv_window_lse, as in the bench, and feed the one-sweep
    scoring. Every head is checked by its saliency mass, sampled heads against the
    oracle's exact softmax saliency and priorities one by one."""
    import torch

    from paper_2609_22158_amd import binding as B
    from synth import make_workload

    w = make_workload("l32_32k", 233)
    g = HipRun(w)
    log("[full l32_32k lse-fed] gpu window LSE and one sweep")
    ws = torch.empty(g.pb.saliency_workspace_bytes(), dtype=torch.uint8, device="cuda")
    lse = B.window_lse(g.pb, g.q, g.k, g.params, workspace=ws)
    sc = g.score(lse=lse, want_saliency=True)
    torch.cuda.synchronize()
    R = w.window * w.group
    A = sc["saliency"].cpu().numpy()
    np.testing.assert_allclose(A.sum(axis=2), R, rtol=1e-4)
    heads = [(0, 3), (17, 0), (31, 6)]
    log("[full l32_32k lse-fed] oracle on sampled heads")
    o = run_oracle(w, g.budget, g.params, heads=heads)
    P = sc["scores"].cpu().numpy()
    for l, h in heads:
        close(A[l, h], o["A"][(0, l, h)], f"A{(l, h)} lse-fed")
        close(P[l, h], o["P"][(0, l, h)], f"P{(l, h)} lse-fed")


def test_full_size_shared_configuration():
    """The bench's --shared-layers 3 configuration at full size: the summed saliency of
    the last 3 layers (24 KV heads x 32k tokens), the single priority row, its ranking
    and the gather of all 32 layers x 8 heads, against the oracle's compress_shared."""
    import torch

    from paper_2609_22158_amd import binding as B
    from synth import make_workload
    from tests.gpu_cases import oracle_utilities

    w = make_workload("l32_32k", 233)
    g = HipRun(w)
    log("[full l32_32k shared] gpu pass")
    sc = B.score_shared(g.pb, g.q, g.k, g.sid, g.prot, g.util, g.params, last_layers=3,
                        want_saliency=True)
    torch.cuda.synchronize()
    log("[full l32_32k shared] oracle")
    o = O.compress_shared(w.q_win, w.k, None, w.cu_seqlens, w.step_ids, w.protected, w.cu_steps,
                          oracle_utilities(w), g.budget, oracle_params(g.params), last_layers=3,
                          want_kv=False)
    A = sc["saliency"].cpu().numpy()
    P = sc["scores"].cpu().numpy()
    close(A, o["A"][0], "A shared full")
    close(P, o["P"][0], "P shared full")
    mass = 3 * w.num_kv_heads * w.window * w.group
    assert abs(A.sum() - mass) < 1e-3 * mass
    # selection on the oracle's priorities (fp32) and the gather of every layer and head
    P32 = o["P"][0].astype(np.float32)
    sel = B.select_shared(g.pb, torch.from_numpy(P32).cuda(), g.prot, g.sid, g.budget)
    idx, cu = sel["idx"], sel["cu_retained"]
    rows = ref_rows(w, g.budget)[0]
    k_hat, v_hat = B.compact_shared(g.pb, g.k, g.v, idx, cu, rows)
    torch.cuda.synchronize()
    want = O.select_retained(P32, w.protected == 0, g.budget)
    got = idx.cpu().numpy()[:rows]
    assert np.array_equal(got, want)
    kh = k_hat.view(torch.int16).cpu().numpy().view(np.uint16)
    for l, h in [(0, 0), (16, 4), (31, 7)]:
        assert np.array_equal(kh[l, h], w.k[l, h][want]), (l, h)
