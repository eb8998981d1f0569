"""Property-based checks of the oracle (Hypothesis), on tiny random inputs.

Each property is fixed by the paper's definitions or by plain mathematics,
not by the oracle's own code: the softmax rows of the window attention sum to
one (Sec. 5.2), the retained set is the protected tokens plus the top-B by
(priority desc, position asc) (Alg. 1 phase 3, eq. problem), the utility is
clipped to [0, S_max] (eq. step-score), pooling is a zero-padded moving
average (Sec. 5.2) and the budget rule is B = max(1, floor(rho N)).
"""
import math

import numpy as np
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle as O

SETTINGS = settings(max_examples=60, deadline=None, derandomize=True)


def _brute_select(P, prun, B):
    """Pure-Python reading of the ranking: sorted() on (-P, i) over the prunable tokens."""
    cand = [i for i in range(len(P)) if prun[i]]

    def key(i):
        x = float(P[i])
        if math.isnan(x):
            x = -math.inf
        return (-x, i)

    take = sorted(cand, key=key)[:min(B, len(cand))]
    return sorted(set(take) | {i for i in range(len(P)) if not prun[i]})


_score = st.one_of(st.sampled_from([0.0, -0.0, 0.25, 0.5, 1.0, float("nan"), -1.0]),
                   st.floats(-4.0, 4.0, allow_nan=False))


@SETTINGS
@given(data=st.data())
def test_select_is_protected_plus_top_b(data):
    n = data.draw(st.integers(0, 60))
    P = np.array(data.draw(st.lists(_score, min_size=n, max_size=n)), dtype=np.float64)
    prun = np.array(data.draw(st.lists(st.booleans(), min_size=n, max_size=n)), dtype=bool)
    B = data.draw(st.integers(0, n + 3))
    idx = O.select_retained(P, prun, B)
    assert list(idx) == _brute_select(P, prun, B)
    assert all(b > a for a, b in zip(idx[:-1], idx[1:]))  # ascending positions
    assert int(prun[idx].sum()) == min(B, int(prun.sum()))  # exactly min(B, N_pr) prunable
    assert set(np.nonzero(~prun)[0]) <= set(idx.tolist())  # protected always kept


@SETTINGS
@given(W=st.integers(1, 4), G=st.integers(1, 3), n=st.integers(1, 12), d=st.integers(1, 6),
       causal=st.booleans(), seed=st.integers(0, 2**31 - 1))
def test_saliency_mass_is_the_number_of_rows_that_see_a_key(W, G, n, d, causal, seed):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(W * G, d)) * 2.0
    k = rng.normal(size=(n, d)) * 2.0
    vis = O.visible_keys(n, W, G, causal)
    A = O.window_saliency(q, k, 1.0 / math.sqrt(d), vis)
    rows_seeing = int(vis.any(axis=1).sum())
    assert (A >= 0).all()
    assert abs(A.sum() - rows_seeing) < 1e-9 * max(1, rows_seeing)
    # a key no row sees gets nothing
    assert (A[~vis.any(axis=0)] == 0).all()


@SETTINGS
@given(W=st.integers(1, 3), G=st.integers(1, 3), n=st.integers(1, 10), d=st.integers(1, 5),
       causal=st.booleans(), seed=st.integers(0, 2**31 - 1))
def test_saliency_from_row_lse_equals_per_row_softmax(W, G, n, d, causal, seed):
    """With each row's log-sum-exp written out by hand in pure Python, the LSE-fed
    saliency equals the column sums of the explicit per-row softmax."""
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(W * G, d))
    k = rng.normal(size=(n, d))
    scale = 1.0 / math.sqrt(d)
    vis = O.visible_keys(n, W, G, causal)
    lse, probs = [], []
    for r in range(W * G):
        z = [scale * sum(q[r, c] * k[i, c] for c in range(d)) for i in range(n)]
        seen = [z[i] for i in range(n) if vis[r, i]]
        if seen:
            m = max(seen)
            tot = sum(math.exp(x - m) for x in seen)
            lse.append(m + math.log(tot))
            probs.append([math.exp(z[i] - m) / tot if vis[r, i] else 0.0 for i in range(n)])
        else:
            lse.append(-math.inf)
            probs.append([0.0] * n)
    want = [sum(probs[r][i] for r in range(W * G)) for i in range(n)]
    got = O.window_saliency_from_lse(q, k, scale, np.array(lse), vis)
    assert np.allclose(got, want, rtol=1e-12, atol=1e-12)


@SETTINGS
@given(n=st.integers(1, 40), kk=st.sampled_from([1, 3, 5, 7, 9]), seed=st.integers(0, 2**31 - 1))
def test_pooling_is_zero_padded_moving_average(n, kk, seed):
    rng = np.random.default_rng(seed)
    A = rng.random(n)
    prun = rng.random(n) > 0.3
    T = O.pooled_saliency(A, prun, kk)
    h = kk // 2
    for i in range(n):
        want = sum(A[j] for j in range(max(0, i - h), min(n, i + h + 1)) if prun[j]) / kk
        assert abs(T[i] - want) < 1e-12


@SETTINGS
@given(data=st.data())
def test_step_utility_stays_in_its_clip_range(data):
    n = data.draw(st.integers(1, 8))
    unit = st.floats(0.0, 1.0)
    valid = data.draw(st.lists(st.sampled_from([0.0, 1.0]), min_size=n, max_size=n))
    gain = data.draw(st.lists(unit, min_size=n, max_size=n))
    red = data.draw(st.lists(unit, min_size=n, max_size=n))
    sims = np.array(data.draw(st.lists(unit, min_size=n * n, max_size=n * n))).reshape(n, n)
    p = O.Params()
    r, c, S = O.run_step_updates(valid, gain, red, sims, p)
    assert (S >= 0).all() and (S <= p.s_max).all()
    assert (c >= 0).all() and (c <= np.arange(n)[::-1] + 1e-12).all()  # c_k gains <= 1 per later step
    # the newest step has had no reuse yet, so its score is the clipped completion score
    assert abs(S[-1] - min(max(p.w_r * min(max(r[-1], p.r_min), p.r_max), 0.0), p.s_max)) < 1e-12


@SETTINGS
@given(rho=st.floats(0.0, 1.0), n=st.integers(0, 100000))
def test_budget_rule(rho, n):
    B = O.budget_from_ratio(rho, n)
    assert B >= 1 and B <= max(1, n)
    # the largest whole number of tokens within the ratio, but never none
    assert B == 1 or B <= rho * n + 1e-9
    assert B + 1 > rho * n - 1e-9
