"""Causal-tail visibility and the LSE-fed single sweep (App. C.2), HIP path vs the oracle.

The row log-sum-exps fed to the GPU come from the oracle (fp64, cast to
fp32), as a prefill's attention would report them; the oracle computes the
saliency from the very same fp32 values. Tolerances as for scores: 2e-3
relative (+1e-7 of the head's max); a row LSE within 2e-3 absolute, which
bounds the relative error it induces in that row's probabilities.
"""
import numpy as np
import pytest

from paper_2609_22158_amd import binding as B
from tests.gpu_cases import HipRun, close, log, oracle_lse, reduced, run_oracle

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": dict(name="tiny"),
    # d = 64 with W * G = 64 rows: 128-key tiles, several per chunk in every plan (16
    # layers fill the chip with multi-tile chunks), both tiles of a barrier summed
    "tiny_long": dict(name="tiny", num_layers=16, seqlens=[20000, 3001]),
    "l1_tail3001": dict(name="l1_8k", seqlens=[3001]),
    # short sequences: N = 1 and 130 < W * G rows; N = 0; a causal tail spanning tiles
    "ragged_g7": dict(name="ragged16", num_layers=2, seqlens=[2500, 700, 130, 1, 0, 4097],
                      protected_len=64),
    # W = 64 (W * G = 256 rows): the tail spans two 32-key tiles
    "l32_w64": dict(name="l32_32k", num_layers=1, seqlens=[3333, 64, 40], num_steps=12,
                    protected_len=16),
    # W = 80 at G = 7: 560 window rows in three groups (256, 256, 48 rows; the last
    # group on the 64-row tiling), each group's tail masked against its own rows
    "ragged_w80": dict(name="ragged16", num_layers=1, window=80, seqlens=[2000, 70, 1, 900],
                       protected_len=32),
}

_w = {}


def _work(cid):
    if cid not in _w:
        spec = dict(CASES[cid])
        _w[cid] = reduced(spec.pop("name"), **spec)
    return _w[cid]


def _heads(w):
    for s in range(w.num_seqs):
        a, b = int(w.cu_seqlens[s]), int(w.cu_seqlens[s + 1])
        for l in range(w.num_layers):
            for h in range(w.num_kv_heads):
                yield s, l, h, a, b


def _compare(w, sc, o, what):
    P = sc["scores"].cpu().numpy()
    A = sc["saliency"].cpu().numpy()
    for s, l, h, a, b in _heads(w):
        close(A[l, h, a:b], o["A"][(s, l, h)], f"{what} A{(s, l, h)}")
        close(P[l, h, a:b], o["P"][(s, l, h)], f"{what} P{(s, l, h)}")


@pytest.mark.parametrize("cid", list(CASES))
def test_causal_two_sweeps_match_oracle(cid):
    w = _work(cid)
    g = HipRun(w, params=B.Params(causal_tail=1))
    log(f"[causal {cid}] seqlens={w.seqlens} W={w.window} G={w.group}")
    sc = g.score(want_saliency=True)
    o = run_oracle(w, g.budget, g.params)
    _compare(w, sc, o, "causal")
    A = sc["saliency"].cpu().numpy()
    for s, l, h, a, b in _heads(w):  # rows that see a key each give one unit of mass
        if b > a:
            seen = min(b - a, w.window) * w.group
            assert abs(A[l, h, a:b].sum() - seen) < 1e-3 * seen


@pytest.mark.parametrize("causal", [0, 1])
@pytest.mark.parametrize("cid", list(CASES))
def test_window_lse_matches_oracle(cid, causal):
    w = _work(cid)
    g = HipRun(w, params=B.Params(causal_tail=causal), want_v=False)
    log(f"[window_lse {cid} causal={causal}]")
    got = B.window_lse(g.pb, g.q, g.k, g.params).cpu().numpy()
    want = oracle_lse(w, bool(causal))
    fin = np.isfinite(want)
    assert np.array_equal(np.isneginf(got), np.isneginf(want)), "rows without keys differ"
    assert fin.sum() + np.isneginf(want).sum() == want.size
    err = np.abs(got[fin] - want[fin])
    assert err.max() <= 2e-3, f"worst row LSE error {err.max():.3e}"


@pytest.mark.parametrize("causal", [0, 1])
@pytest.mark.parametrize("cid", list(CASES))
def test_lse_fed_single_sweep_matches_oracle(cid, causal):
    w = _work(cid)
    g = HipRun(w, params=B.Params(causal_tail=causal), want_v=False)
    lse32 = oracle_lse(w, bool(causal)).astype(np.float32)  # what a prefill would hand over
    log(f"[lse-fed {cid} causal={causal}]")
    sc = g.score(lse=g.lse_tensor(lse32), want_saliency=True)
    o = run_oracle(w, g.budget, g.params, lse_win=lse32.astype(np.float64))
    _compare(w, sc, o, f"lse-fed causal={causal}")


def test_lse_fed_with_gpu_lse_equals_two_sweeps():
    """stepkv_window_lse followed by stepkv_saliency_from_lse reproduces stepkv_saliency."""
    w = _work("l1_tail3001")
    g = HipRun(w, want_v=False)
    lse = B.window_lse(g.pb, g.q, g.k, g.params)
    a1 = B.saliency_from_lse(g.pb, g.q, g.k, lse, g.params).cpu().numpy()
    a2 = B.saliency(g.pb, g.q, g.k, g.params).cpu().numpy()
    for s, l, h, a, b in _heads(w):
        close(a1[l, h, a:b], a2[l, h, a:b].astype(np.float64), f"A{(s, l, h)}")


def test_lse_shift_scales_rows():
    """Raising every row's LSE by ln 2 halves every saliency (a property at any size)."""
    w = _work("tiny")
    g = HipRun(w, want_v=False)
    lse = B.window_lse(g.pb, g.q, g.k, g.params)
    a1 = B.saliency_from_lse(g.pb, g.q, g.k, lse, g.params).cpu().numpy()
    a2 = B.saliency_from_lse(g.pb, g.q, g.k, lse + float(np.log(2.0)), g.params).cpu().numpy()
    np.testing.assert_allclose(a2, 0.5 * a1, rtol=2e-6, atol=1e-12)
