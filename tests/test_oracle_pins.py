"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test names the passage of the paper whose definition it pins and what
fixes the expected value: a hand-evaluated closed form, an invariant, a
library routine the oracle does not call, or a special case of the method
that reduces to something simpler.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle as O
from synth import f32_to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bits(x):
    return f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


# ------------------------------------------------------------- bf16 decoding
# Hand-decoded bf16 bit patterns: sign bit 15, exponent bits 14-7 (bias 127),
# mantissa bits 6-0; exponent 0 is subnormal (2^-126 * m/128), 255 is inf/NaN.
BF16_HAND = [
    (0x3F80, 1.0),
    (0x3F00, 0.5),
    (0xC000, -2.0),
    (0xC020, -2.5),  # exponent 128, mantissa 0x20 -> -(1 + 32/128) * 2
    (0x4049, 3.140625),  # exponent 128, mantissa 73 -> (1 + 73/128) * 2
    (0x0080, math.ldexp(1.0, -126)),  # smallest normal
    (0x0001, math.ldexp(1.0, -133)),  # smallest subnormal: 2^-126 / 128
    (0x807F, -math.ldexp(127.0, -133)),  # largest negative subnormal
    (0x7F7F, math.ldexp(255.0, 120)),  # largest finite: (255/128) * 2^127
    (0x7F80, math.inf),
    (0xFF80, -math.inf),
    (0x0000, 0.0),
]


def test_decode_bf16_hand_bit_patterns():
    """bf16 is the top half of an IEEE binary32 word; every value is exact in fp64."""
    raw = np.array([b for b, _ in BF16_HAND], dtype=np.uint16)
    got = O.decode_bf16(raw)
    assert got.dtype == np.float64
    for (b, want), g in zip(BF16_HAND, got):
        assert g == want, f"0x{b:04X}: {g!r} != {want!r}"
    neg_zero = O.decode_bf16(np.array([0x8000], dtype=np.uint16))[0]
    assert neg_zero == 0.0 and math.copysign(1.0, neg_zero) == -1.0
    for b in (0x7FC0, 0xFFC1, 0x7F81):  # quiet, negative and signalling NaN payloads
        assert math.isnan(O.decode_bf16(np.array([b], dtype=np.uint16))[0])
    # the shape is kept and element order follows the array, not the bytes
    grid = raw[:12].reshape(3, 4)
    np.testing.assert_array_equal(O.decode_bf16(grid), got[:12].reshape(3, 4))
    # the round trip through the generators' RNE encoder on values exact in bf16
    vals = np.array([w for _, w in BF16_HAND if math.isfinite(w)], dtype=np.float32)
    np.testing.assert_array_equal(O.decode_bf16(bits(vals)), vals.astype(np.float64))


# ------------------------------------------------------------- step utility
def _golden_cases():
    with open(os.path.join(GOLDEN, "step_utility.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _golden_cases(), ids=lambda c: c["name"])
def test_step_utility_hand_values(case):
    """eq. reward / eq. reuse / eq. step-score in Algorithm 1's order (Sec. 5.1, App. C.3)."""
    p = O.Params(**case["params"])
    _, _, S = O.run_step_updates(case["valid"], case["gain"], case["red"],
                                 np.array(case["obs_sim"], dtype=np.float64), p)
    expect = [eval(e, {"log": math.log}) for e in case["expect_S"]]
    np.testing.assert_allclose(S, expect, rtol=0, atol=1e-12)


def test_reuse_accumulator_bounds():
    """App. C.1: each reuse increment lies in [0, 1], so c_k >= 0 and grows by <= 1 a boundary."""
    rng = np.random.default_rng(0)
    n = 40
    sim = np.tril(rng.random((n, n)), -1)
    _, c, S = O.run_step_updates(np.ones(n), rng.random(n), rng.random(n), sim, O.Params())
    assert (c >= 0).all()
    for k in range(n):
        assert c[k] <= (n - 1 - k) + 1e-12  # one increment per later boundary
    assert (S >= 0).all() and (S <= 8).all()


def test_budget_from_ratio():
    """eq. problem: B_t = max(1, floor(rho N_t)); rho N computed in fp must not drop a unit."""
    assert O.budget_from_ratio(0.2, 1000) == 200
    assert O.budget_from_ratio(0.2, 3) == 1  # floor(0.6) = 0 -> max(1, 0)
    assert O.budget_from_ratio(0.29, 100) == 29  # 0.29*100 = 28.999999999999996 in fp64
    assert O.budget_from_ratio(0.5, 7) == 3


# ------------------------------------------------------------- saliency
def _rows_keys(W, G, d, N, seed):
    rng = np.random.default_rng(seed)
    q = O.decode_bf16(bits(rng.standard_normal((W * G, d))))
    k = O.decode_bf16(bits(rng.standard_normal((N, d)) / math.sqrt(d)))
    return q, k


def test_saliency_zero_queries_is_uniform():
    """With Q = 0 every row-softmax is uniform, so A_i = W*G/N exactly."""
    _, k = _rows_keys(4, 3, 64, 37, 1)
    A = O.window_saliency(np.zeros((12, 64)), k, 0.125)
    np.testing.assert_allclose(A, np.full(37, 12 / 37), rtol=1e-15)


def test_saliency_two_level_closed_form():
    """Keys on one axis give two logit levels; the softmax has a closed form."""
    d, N, W, G = 64, 50, 8, 2
    scale = 1.0 / math.sqrt(d)
    c, a, b = 3.0, 1.5, -0.5
    q = np.zeros((W * G, d))
    q[:, 0] = c
    k = np.zeros((N, d))
    hi = np.arange(N) % 5 == 0  # 10 keys at level a, 40 at level b
    k[hi, 0] = a
    k[~hi, 0] = b
    A = O.window_saliency(q, k, scale)
    za, zb = c * a * scale, c * b * scale
    den = 10 * math.exp(za) + 40 * math.exp(zb)
    expect = np.where(hi, W * G * math.exp(za) / den, W * G * math.exp(zb) / den)
    np.testing.assert_allclose(A, expect, rtol=1e-13)


def test_saliency_matches_library_softmax():
    """A = column sums of softmax(scale Q K^T) (scipy and torch softmax, not the oracle's exp)."""
    q, k = _rows_keys(16, 4, 128, 301, 2)
    scale = 1.0 / math.sqrt(128)
    z = (q @ k.T) * scale
    ref_scipy = scipy.special.softmax(z, axis=1).sum(axis=0)
    ref_torch = torch.softmax(torch.from_numpy(z), dim=1).sum(dim=0).numpy()
    A = O.window_saliency(q, k, scale)
    np.testing.assert_allclose(A, ref_scipy, rtol=1e-12)
    np.testing.assert_allclose(A, ref_torch, rtol=1e-12)


def test_saliency_invariants():
    """A >= 0 and sum_i A_i = W*G (each row-softmax sums to one)."""
    q, k = _rows_keys(32, 4, 128, 999, 3)
    A = O.window_saliency(q, k * 5.0, 1.0 / math.sqrt(128))
    assert (A >= 0).all()
    assert abs(A.sum() - 128) < 1e-10


def test_gqa_row_mapping():
    """Query head h_q reads KV head floor(h_q / G); window row r = w*G + g."""
    W, Hq, Hkv, d = 3, 4, 2, 64
    G = Hq // Hkv
    q = np.zeros((W, Hq, d))
    q[1, 1, 5] = 40.0  # query head 1 -> KV head 0, window slot 1
    rows0 = O.window_rows(q, 0, G)
    rows1 = O.window_rows(q, 1, G)
    assert rows0.shape == (W * G, d)
    assert rows0[1 * G + 1, 5] == 40.0 and np.count_nonzero(rows0) == 1
    assert np.count_nonzero(rows1) == 0
    k = np.zeros((20, d))
    k[7, 5] = 1.0
    A0 = O.window_saliency(rows0, k, 1.0)
    A1 = O.window_saliency(rows1, k, 1.0)
    np.testing.assert_allclose(A1, np.full(20, W * G / 20), rtol=1e-15)
    assert A0.argmax() == 7 and A0[7] > W * G / 20 + 0.9


def test_saliency_brute_force_loops():
    """Pure-Python loops with math.exp on a tiny case (a second, unvectorised reading)."""
    q, k = _rows_keys(4, 2, 64, 23, 4)
    scale = 0.125
    A = [0.0] * 23
    for r in range(8):
        z = [scale * sum(q[r, j] * k[i, j] for j in range(64)) for i in range(23)]
        m = max(z)
        e = [math.exp(x - m) for x in z]
        t = sum(e)
        for i in range(23):
            A[i] += e[i] / t
    np.testing.assert_allclose(O.window_saliency(q, k, scale), A, rtol=1e-12)


# ------------------------------------------------------------- causal tail, saliency from LSE
def test_causal_visibility_rule():
    """Window slot w is the query at position N - W + w and sees keys 0 .. N - W + w."""
    vis = O.visible_keys(10, 4, 2, True)
    assert vis.shape == (8, 10)
    for r in range(8):
        w = r // 2
        assert vis[r].tolist() == [i <= 10 - 4 + w for i in range(10)]
    assert O.visible_keys(10, 4, 2, False).all()


def test_causal_saliency_brute_force_loops():
    """Pure-Python loops with math.exp over each row's visible keys only."""
    W, G, d, n = 4, 2, 64, 23
    q, k = _rows_keys(W, G, d, n, 5)
    scale = 0.125
    A = [0.0] * n
    for r in range(W * G):
        w = r // G
        seen = [i for i in range(n) if i <= n - W + w]
        z = {i: scale * sum(q[r, j] * k[i, j] for j in range(d)) for i in seen}
        m = max(z.values())
        t = sum(math.exp(x - m) for x in z.values())
        for i in seen:
            A[i] += math.exp(z[i] - m) / t
    got = O.window_saliency(q, k, scale, O.visible_keys(n, W, G, True))
    np.testing.assert_allclose(got, A, rtol=1e-12)


def test_causal_single_slot_sees_everything():
    """W = 1: the last query sees every key, so the causal tail changes nothing."""
    q, k = _rows_keys(1, 4, 128, 77, 6)
    scale = 1.0 / math.sqrt(128)
    np.testing.assert_allclose(O.window_saliency(q, k, scale, O.visible_keys(77, 1, 4, True)),
                               O.window_saliency(q, k, scale), rtol=1e-14)


def test_causal_full_window_is_causal_attention():
    """N = W, G = 1: column sums of a lower-triangular softmax (torch masked softmax)."""
    n = 19
    q, k = _rows_keys(n, 1, 64, n, 7)
    scale = 0.125
    z = torch.from_numpy((q @ k.T) * scale)
    z = z.masked_fill(torch.triu(torch.ones(n, n, dtype=torch.bool), diagonal=1), -math.inf)
    ref = torch.softmax(z, dim=1).sum(dim=0).numpy()
    got = O.window_saliency(q, k, scale, O.visible_keys(n, n, 1, True))
    np.testing.assert_allclose(got, ref, rtol=1e-12)
    assert abs(got[-1] - float(torch.softmax(z, dim=1)[-1, -1])) < 1e-14  # only the last row sees it


def test_causal_rows_without_keys_contribute_nothing():
    """N < W: slots w < W - N see no key; the sum of A counts only the other N*G rows."""
    W, G, n = 8, 2, 5
    q, k = _rows_keys(W, G, 64, n, 8)
    vis = O.visible_keys(n, W, G, True)
    assert (~vis[: (W - n) * G]).all() and vis[(W - n) * G:].any(axis=1).all()
    A = O.window_saliency(q, k, 0.125, vis)
    assert abs(A.sum() - n * G) < 1e-12
    lse = O.window_row_lse(q, k, 0.125, vis)
    assert np.isneginf(lse[: (W - n) * G]).all() and np.isfinite(lse[(W - n) * G:]).all()


@pytest.mark.parametrize("causal", [False, True])
def test_row_lse_matches_scipy_logsumexp(causal):
    """Row log-sum-exp over the visible keys equals scipy's logsumexp on the same logits."""
    W, G, n = 16, 4, 300
    q, k = _rows_keys(W, G, 128, n, 9)
    scale = 1.0 / math.sqrt(128)
    vis = O.visible_keys(n, W, G, causal)
    z = (q @ k.T) * scale
    ref = np.array([scipy.special.logsumexp(z[r][vis[r]]) for r in range(W * G)])
    np.testing.assert_allclose(O.window_row_lse(q, k, scale, vis), ref, rtol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_saliency_from_exact_lse_equals_softmax_sums(causal):
    """Fed the exact row LSE (from scipy), the one-sweep form gives the two-sweep A."""
    W, G, n = 16, 4, 300
    q, k = _rows_keys(W, G, 128, n, 10)
    scale = 1.0 / math.sqrt(128)
    vis = O.visible_keys(n, W, G, causal)
    z = (q @ k.T) * scale
    lse = np.array([scipy.special.logsumexp(z[r][vis[r]]) for r in range(W * G)])
    ref = scipy.special.softmax(np.where(vis, z, -np.inf), axis=1).sum(axis=0)
    np.testing.assert_allclose(O.window_saliency_from_lse(q, k, scale, lse, vis), ref, rtol=1e-12)
    np.testing.assert_allclose(O.window_saliency(q, k, scale, vis), ref, rtol=1e-12)


def test_saliency_from_lse_shift():
    """Raising row r's LSE by delta_r scales that row's contribution by exp(-delta_r)."""
    W, G, n = 8, 2, 120
    q, k = _rows_keys(W, G, 64, n, 11)
    scale = 0.125
    lse = O.window_row_lse(q, k, scale)
    delta = np.linspace(-2.0, 3.0, W * G)
    p = O.window_attention(q, k, scale)
    np.testing.assert_allclose(O.window_saliency_from_lse(q, k, scale, lse + delta),
                               (p * np.exp(-delta)[:, None]).sum(axis=0), rtol=1e-12)


# ------------------------------------------------------------- pooling, normalisation
def test_pool_constant_closed_form():
    """Constant A on prunable tokens: interior T = A, an edge with e missing taps gives A(k-e)/k."""
    n, k = 30, 7
    A = np.full(n, 2.0)
    T = O.pooled_saliency(A, np.ones(n, bool), k)
    np.testing.assert_allclose(T[3:-3], 2.0, rtol=1e-15)
    for e in range(1, 4):
        np.testing.assert_allclose(T[3 - e], 2.0 * (k - e) / k, rtol=1e-15)
        np.testing.assert_allclose(T[n - 4 + e], 2.0 * (k - e) / k, rtol=1e-15)


def test_pool_impulse_response_and_protected_mask():
    """An impulse spreads A_j/k over exactly [j-3, j+3]; protected tokens contribute nothing."""
    n = 40
    A = np.zeros(n)
    A[20] = 7.0
    A[2] = 100.0  # protected below
    prun = np.ones(n, bool)
    prun[:5] = False
    T = O.pooled_saliency(A, prun, 7)
    expect = np.zeros(n)
    expect[17:24] = 1.0
    np.testing.assert_allclose(T, expect, rtol=1e-15, atol=0)


def test_normalisation_uses_prunable_max():
    """T_hat in [0, 1] with 1 at the prunable argmax; a large protected value does not flatten it."""
    T = np.array([50.0, 1.0, 4.0, 2.0, 0.0])
    prun = np.array([False, True, True, True, True])
    Th = O.normalised_saliency(T, prun)
    np.testing.assert_allclose(Th[1:], [0.25, 1.0, 0.5, 0.0], rtol=1e-15)
    assert (O.normalised_saliency(np.zeros(4), np.ones(4, bool)) == 0).all()


# ------------------------------------------------------------- priority and selection
def test_priority_range_and_dominance():
    """App. C.1: Score in [0, alpha H_max + beta U_max]; the step preference flips exactly
    where alpha (H_i - H_j) = beta (U_s(j) - U_s(i))."""
    S = np.array([0.5, 1.0])
    sid = np.array([0, 1])
    prun = np.ones(2, bool)
    alpha, beta = 0.2, 0.8
    # token 0 (step utility 0.5) out-salients token 1 (utility 1.0) by dH
    # threshold dH* = beta (1.0 - 0.5) / alpha = 2 > 1, so within [0,1] the step wins
    P = O.priority(np.array([1.0, 0.0]), sid, S, prun, alpha, beta)
    assert P[1] > P[0]
    P = O.priority(np.array([1.0, 0.0]), sid, np.array([0.5, 0.6]), prun, alpha, beta)
    # dH = 1 > beta*0.1/alpha = 0.4 -> token saliency wins
    assert P[0] > P[1]
    rng = np.random.default_rng(5)
    Th = rng.random(100)
    Sr = rng.random(10) * 8
    P = O.priority(Th, rng.integers(0, 10, 100), Sr, np.ones(100, bool), alpha, beta)
    assert P.min() >= 0 and P.max() <= alpha * 1 + beta * 8


def _brute_select(P, prun, B):
    """Python's sorted() on (-P, i): a different sort routine from the oracle's lexsort."""
    cand = [i for i in range(len(P)) if prun[i]]

    def key(i):
        x = float(P[i])
        if math.isnan(x):
            x = -math.inf
        return (-x, i)

    take = sorted(cand, key=key)[:min(B, len(cand))]
    return sorted(set(take) | {i for i in range(len(P)) if not prun[i]})


@pytest.mark.parametrize("seed", range(6))
def test_select_matches_python_sorted(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 300))
    P = np.round(rng.random(n) * 5) / 5  # many exact ties
    P[rng.random(n) < 0.05] = np.nan
    P[rng.random(n) < 0.05] = -0.0
    prun = rng.random(n) > 0.2
    B = int(rng.integers(1, n + 5))
    idx = O.select_retained(P, prun, B)
    assert list(idx) == _brute_select(P, prun, B)
    assert (np.diff(idx) > 0).all()
    assert int(prun[idx].sum()) == min(B, int(prun.sum()))
    assert set(np.nonzero(~prun)[0]) <= set(idx)


def test_select_alpha_zero_takes_whole_steps():
    """alpha = 0 (no token score, Table 3): whole steps in descending S, lowest positions first."""
    sid = np.repeat(np.arange(4), 10)
    S = np.array([0.3, 1.2, 0.7, 1.2])
    prun = np.ones(40, bool)
    P = O.priority(np.random.default_rng(1).random(40), sid, S, prun, 0.0, 0.8)
    idx = O.select_retained(P, prun, 25)
    expect = list(range(10, 20)) + list(range(30, 40)) + list(range(20, 25))
    assert list(idx) == sorted(expect)


def test_select_beta_zero_is_saliency_topk():
    """beta = 0 (no step score, Table 3): the plain top-B of T_hat."""
    rng = np.random.default_rng(2)
    Th = rng.random(200)
    sid = rng.integers(0, 5, 200)
    prun = np.ones(200, bool)
    P = O.priority(Th, sid, rng.random(5), prun, 0.2, 0.0)
    idx = O.select_retained(P, prun, 30)
    assert set(idx) == set(np.argsort(-Th)[:30])


def test_select_all_equal_and_budget_edges():
    prun = np.array([0, 0, 1, 1, 1, 1, 1], bool)
    P = np.zeros(7)
    assert list(O.select_retained(P, prun, 2)) == [0, 1, 2, 3]
    assert list(O.select_retained(P, prun, 99)) == list(range(7))
    assert list(O.select_retained(P, np.zeros(7, bool), 3)) == list(range(7))  # all protected
    assert list(O.select_retained(P, ~np.zeros(7, bool), 0)) == []


@pytest.mark.parametrize("seed", range(4))
def test_retained_count_is_the_selection_size(seed):
    """eq. problem with exactly min(B, N_pr) kept: the count equals the size of the
    selection itself (which is pinned against Python's sorted()), protected tokens anywhere."""
    rng = np.random.default_rng(40 + seed)
    for _ in range(20):
        n = int(rng.integers(0, 120))
        prun = rng.random(n) > 0.3
        B = int(rng.integers(1, 150))
        P = rng.random(n)
        assert O.retained_count(n, int((~prun).sum()), B) == len(O.select_retained(P, prun, B))
    assert O.retained_count(10, 10, 5) == 10 and O.retained_count(0, 0, 3) == 0
    assert O.retained_count(1000, 512, 1024) == 1000 and O.retained_count(4096, 512, 2048) == 2560


def test_kept_per_step_sums_to_kept():
    rng = np.random.default_rng(3)
    sid = np.concatenate([np.full(5, -1), np.repeat(np.arange(6), 9)])
    prun = sid >= 0
    P = O.priority(rng.random(59), sid, rng.random(6), prun, 0.2, 0.8)
    idx = O.select_retained(P, prun, 17)
    kept = O.kept_per_step(idx, sid, prun, 6)
    assert kept.sum() == 17
    st = O.step_statistics(rng.random(59), sid, prun, 6)
    assert (st["count"] == 9).all()


def test_kept_per_step_hand_values():
    """Retained prunable tokens per step (the per-step view behind Figs. 2 and 8), worked
    out by hand: protected tokens, a prunable token with id -1 and one with an id past the
    step count are retained but counted in no step."""
    #            pos: 0   1   2  3  4  5  6  7  8  9  10 11
    sid = np.array([-1, -1, 0, 0, 1, 1, 1, 2, 5, 0, 2, -1])
    prun = np.array([0, 1, 1, 1, 1, 1, 1, 1, 1, 0, 1, 1], bool)
    idx = np.array([0, 1, 3, 4, 6, 7, 8, 9, 10])
    # step 0: pos 3 (pos 9 is protected); step 1: pos 4 and 6; step 2: pos 7 and 10;
    # pos 0 (protected, -1), 1 (prunable, -1) and 8 (id 5 >= 3) count nowhere
    np.testing.assert_array_equal(O.kept_per_step(idx, sid, prun, 3), [1, 2, 2])
    np.testing.assert_array_equal(O.kept_per_step(idx, sid, prun, 6), [1, 2, 2, 0, 0, 1])
    np.testing.assert_array_equal(O.kept_per_step(idx[:0], sid, prun, 3), [0, 0, 0])
    # every prunable token of steps 0..2 retained: the counts are the step lengths
    all_idx = np.arange(12)
    np.testing.assert_array_equal(O.kept_per_step(all_idx, sid, prun, 3), [2, 3, 2])


def test_step_statistics_hand_values():
    """Per-step diagnostics (the token counts and saliency mass behind Figs. 2 and 8) on a
    hand-worked example: a protected token, an id of -1 and an id past the step count are
    left out; values worked out by hand."""
    T_hat = np.array([0.5, 0.2, 0.9, 0.1, 0.4, 0.7, 0.3])
    sid = np.array([0, 0, 1, 1, -1, 5, 1])
    prun = np.array([True, False, True, True, True, True, True])
    st = O.step_statistics(T_hat, sid, prun, 2)
    assert list(st["count"]) == [1, 3]
    assert np.allclose(st["max"], [0.5, 0.9], rtol=0, atol=1e-15)
    assert np.allclose(st["sum"], [0.5, 1.3], rtol=0, atol=1e-15)


# ------------------------------------------------------------- compaction, decode
def test_compact_is_row_gather():
    rng = np.random.default_rng(4)
    K = rng.integers(0, 65535, (50, 8), dtype=np.uint16)
    V = rng.integers(0, 65535, (50, 8), dtype=np.uint16)
    idx = np.array([0, 3, 4, 17, 49])
    kh, vh = O.compact(K, V, idx)
    for j, i in enumerate(idx):
        assert (kh[j] == K[i]).all() and (vh[j] == V[i]).all()


def test_decode_attention_matches_torch_sdpa():
    rng = np.random.default_rng(6)
    K = rng.standard_normal((33, 64))
    V = rng.standard_normal((33, 64))
    q = rng.standard_normal(64)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, None, None], torch.from_numpy(K)[None, None],
        torch.from_numpy(V)[None, None]).numpy().reshape(-1)
    np.testing.assert_allclose(O.decode_attention(q, K, V, 1 / 8), ref, rtol=1e-12)
    # one retained row: the output is that value row
    np.testing.assert_allclose(O.decode_attention(q, K[:1], V[:1], 1 / 8), V[0], rtol=1e-15)


# ------------------------------------------------------------- batched sequences
def _batch_case(lens=(70, 0, 1, 95), steps=(5, 1, 1, 7), prot_len=(6, 0, 1, 9), L=2, Hkv=2,
                G=3, W=4, d=64, seed=21):
    """A ragged batch in the library's layout: sequences concatenated along the token axis,
    step utilities concatenated along cu_steps, one q_win / lse_win slice per sequence."""
    rng = np.random.default_rng(seed)
    nseq, ntot = len(lens), sum(lens)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    cs = np.concatenate([[0], np.cumsum(steps)]).astype(np.int64)
    q = bits(rng.standard_normal((L, nseq, W, Hkv * G, d)))
    k = bits(rng.standard_normal((L, Hkv, ntot, d)) / math.sqrt(d))
    v = bits(rng.standard_normal((L, Hkv, ntot, d)))
    sid = np.full(ntot, -1, np.int32)
    prot = np.zeros(ntot, np.uint8)
    for s in range(nseq):
        a, b = int(cu[s]), int(cu[s + 1])
        prot[a:a + prot_len[s]] = 1
        n_pr = b - a - prot_len[s]
        if n_pr > 0:
            sid[a + prot_len[s]:b] = np.sort(rng.integers(0, steps[s], n_pr))
    S = rng.uniform(0.0, 1.7, int(cs[-1]))
    lse = rng.normal(2.0, 0.5, (L, nseq, W, Hkv * G))  # not the exact LSE: each row's
    return q, k, v, cu, sid, prot, cs, S, lse          # value changes its contribution


def _alone(case, s):
    """Sequence s of a batch as a one-sequence problem."""
    q, k, v, cu, sid, prot, cs, S, lse = case
    a, b = int(cu[s]), int(cu[s + 1])
    return (q[:, s:s + 1], k[:, :, a:b], v[:, :, a:b], np.array([0, b - a]), sid[a:b],
            prot[a:b], np.array([0, cs[s + 1] - cs[s]]), S[cs[s]:cs[s + 1]], lse[:, s:s + 1])


@pytest.mark.parametrize("mode", ["two-sweep", "lse-fed", "causal"])
def test_compress_batch_equals_each_sequence_alone(mode):
    """eq. problem holds per sequence: on a ragged batch, the pass over the concatenated
    layout (cu_seqlens, cu_steps, the sequence's q_win / lse_win slice) gives for every
    sequence what the pass over that sequence alone gives: P, A, T_hat, idx, kept, K_hat, V_hat."""
    case = _batch_case()
    q, k, v, cu, sid, prot, cs, S, lse = case
    p = O.Params(causal_tail=(mode == "causal"))
    use_lse = mode == "lse-fed"
    batch = O.compress(q, k, v, cu, sid, prot, cs, S, 9, p, want_saliency=True,
                       lse_win=lse if use_lse else None)
    seen = 0
    for s in range(len(cu) - 1):
        q1, k1, v1, cu1, sid1, prot1, cs1, S1, lse1 = _alone(case, s)
        one = O.compress(q1, k1, v1, cu1, sid1, prot1, cs1, S1, 9, p, want_saliency=True,
                         lse_win=lse1 if use_lse else None)
        for l in range(q.shape[0]):
            for h in range(k.shape[1]):
                got, want = (s, l, h), (0, l, h)
                for f in ("P", "A", "T_hat"):
                    np.testing.assert_array_equal(batch[f][got], one[f][want], err_msg=f)
                for f in ("idx", "kept"):
                    np.testing.assert_array_equal(batch[f][got], one[f][want], err_msg=f)
                for f, src in (("k_hat", k1), ("v_hat", v1)):  # an empty cache stores none
                    want_rows = one[f].get(want, src[l, h][one["idx"][want]])
                    np.testing.assert_array_equal(batch[f][got], want_rows, err_msg=f)
                seen += 1
    assert seen == 4 * 2 * 2
    a3 = int(cu[3])
    assert len(batch["idx"][(3, 1, 1)]) == 9 + 9 and batch["idx"][(1, 0, 0)].size == 0
    assert list(batch["idx"][(2, 0, 0)]) == [0]  # one protected token, nothing prunable
    assert batch["kept"][(3, 0, 0)].sum() == 9 and len(batch["kept"][(3, 0, 0)]) == 7
    np.testing.assert_array_equal(batch["k_hat"][(3, 1, 0)],
                                  k[1, 0, a3:][batch["idx"][(3, 1, 0)]])


def test_compress_batch_uses_each_sequences_own_slices():
    """The per-sequence slices are not interchangeable: changing sequence 3's window
    queries, utilities or row LSEs changes sequence 3's result and no other."""
    case = _batch_case()
    q, k, v, cu, sid, prot, cs, S, lse = case
    base = O.compress(q, k, v, cu, sid, prot, cs, S, 9, want_saliency=True, lse_win=lse)
    q2 = q.copy()
    q2[:, 3] = bits(np.random.default_rng(7).standard_normal(q2[:, 3].shape))
    S2 = S.copy()
    S2[cs[3]:cs[4]] = S2[cs[3]:cs[4]][::-1] + 0.05
    lse2 = lse.copy()
    lse2[:, 3] += np.random.default_rng(8).normal(0, 1, lse2[:, 3].shape)
    for kw in ({"q_win": q2}, {"S": S2}, {"lse_win": lse2}):
        args = dict(q_win=q, k=k, v=v, cu_seqlens=cu, step_ids=sid, protected=prot,
                    cu_steps=cs, S=S, budget=9, want_saliency=True, lse_win=lse)
        args.update(kw)
        out = O.compress(**args)
        for key in base["P"]:
            same = np.array_equal(out["P"][key], base["P"][key])
            assert same == (key[0] != 3), (list(kw), key)


@pytest.mark.parametrize("causal", [False, True])
def test_compress_lse_fed_with_library_lse_equals_two_sweeps(causal):
    """App. C.2: given every window row's exact log-sum-exp in the lse_win layout
    [L][S][W][Hq] (scipy's logsumexp over the keys the row sees, per sequence), the
    LSE-fed pass equals the two-sweep pass on every sequence, layer and KV head."""
    q, k, v, cu, sid, prot, cs, S, _ = _batch_case()
    L, nseq, W, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    qf, kf = O.decode_bf16(q), O.decode_bf16(k)
    lse = np.full((L, nseq, W, Hq), -np.inf)
    for l in range(L):
        for s in range(nseq):
            a, b = int(cu[s]), int(cu[s + 1])
            n = b - a
            for w in range(W):
                last = n - W + w if causal else n - 1  # the last key slot w sees
                for hq in range(Hq):
                    if last < 0 or n == 0:
                        continue
                    z = kf[l, hq // G, a:a + last + 1] @ qf[l, s, w, hq] / math.sqrt(d)
                    lse[l, s, w, hq] = scipy.special.logsumexp(z)
    p = O.Params(causal_tail=causal)
    two = O.compress(q, k, v, cu, sid, prot, cs, S, 9, p, want_saliency=True)
    fed = O.compress(q, k, v, cu, sid, prot, cs, S, 9, p, want_saliency=True, lse_win=lse)
    for key in two["P"]:
        np.testing.assert_allclose(fed["A"][key], two["A"][key], rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(fed["P"][key], two["P"][key], rtol=1e-12)
        np.testing.assert_array_equal(fed["idx"][key], two["idx"][key])


# ------------------------------------------------------------- shared-index mode
def _shared_case(L=3, Hkv=2, G=2, W=4, d=64, n=60, n_steps=5, seed=12):
    rng = np.random.default_rng(seed)
    q = bits(rng.standard_normal((L, 1, W, Hkv * G, d)))
    k = bits(rng.standard_normal((L, Hkv, n, d)) / math.sqrt(d))
    v = bits(rng.standard_normal((L, Hkv, n, d)))
    prot = np.zeros(n, np.uint8)
    prot[:6] = 1
    sid = np.concatenate([np.full(6, -1), np.sort(rng.integers(0, n_steps, n - 6))]).astype(np.int32)
    S = rng.uniform(0.0, 1.7, n_steps)
    return q, k, v, np.array([0, n]), sid, prot, np.array([0, n_steps]), S


def test_shared_mode_single_head_is_the_per_head_mode():
    """One layer, one KV head: the shared ranking is the per-head ranking."""
    q, k, v, cu, sid, prot, cs, S = _shared_case(L=1, Hkv=1)
    sh = O.compress_shared(q, k, v, cu, sid, prot, cs, S, 20, last_layers=3)
    ph = O.compress(q, k, v, cu, sid, prot, cs, S, 20, want_saliency=True)
    np.testing.assert_array_equal(sh["idx"][0], ph["idx"][(0, 0, 0)])
    np.testing.assert_allclose(sh["P"][0], ph["P"][(0, 0, 0)], rtol=1e-15)


def test_shared_mode_sums_only_the_last_layers():
    """A sums to (layers used) x Hkv x W x G; layers before the last n have no influence."""
    q, k, v, cu, sid, prot, cs, S = _shared_case(L=4)
    sh = O.compress_shared(q, k, v, cu, sid, prot, cs, S, 20, last_layers=3)
    assert abs(sh["A"][0].sum() - 3 * 2 * 4 * 2) < 1e-10
    q2, k2 = q.copy(), k.copy()
    q2[0] = bits(np.random.default_rng(99).standard_normal(q2[0].shape))  # layer 0 is not used
    k2[0] = bits(np.random.default_rng(98).standard_normal(k2[0].shape))
    sh2 = O.compress_shared(q2, k2, v, cu, sid, prot, cs, S, 20, last_layers=3)
    np.testing.assert_array_equal(sh2["A"][0], sh["A"][0])
    np.testing.assert_array_equal(sh2["idx"][0], sh["idx"][0])
    one = O.compress_shared(q, k, v, cu, sid, prot, cs, S, 20, last_layers=1)
    assert abs(one["A"][0].sum() - 2 * 4 * 2) < 1e-10


def test_shared_mode_pooling_is_linear_over_heads():
    """T_hat of the summed A equals the normalised sum of the per-head pooled T (pooling is linear)."""
    q, k, v, cu, sid, prot, cs, S = _shared_case(L=3)
    sh = O.compress_shared(q, k, v, cu, sid, prot, cs, S, 20, last_layers=3)
    ph = O.compress(q, k, v, cu, sid, prot, cs, S, 20, want_saliency=True)
    prun = prot == 0
    T = sum(O.pooled_saliency(ph["A"][(0, l, h)], prun, 7) for l in range(3) for h in range(2))
    np.testing.assert_allclose(sh["T_hat"][0], T / T[prun].max(), rtol=1e-12)


def test_shared_mode_one_index_set_for_every_head():
    """k_hat / v_hat of every (layer, head) gather the same positions, in order."""
    q, k, v, cu, sid, prot, cs, S = _shared_case(L=3, n=80)
    sh = O.compress_shared(q, k, v, cu, sid, prot, cs, S, 25, last_layers=2)
    idx = sh["idx"][0]
    assert len(idx) == 6 + 25 and (np.diff(idx) > 0).all() and set(range(6)) <= set(idx.tolist())
    for l in range(3):
        for h in range(2):
            np.testing.assert_array_equal(sh["k_hat"][0][l, h], k[l, h][idx])
            np.testing.assert_array_equal(sh["v_hat"][0][l, h], v[l, h][idx])
    # the shared ranking is the top of P by (P desc, position asc), as Python's sorted() orders it
    P = sh["P"][0]
    order = sorted((i for i in range(80) if prot[i] == 0), key=lambda i: (-P[i], i))[:25]
    assert sorted(order) == [int(i) for i in idx if prot[i] == 0]
