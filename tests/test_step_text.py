"""Step signals from text (Sec. 5.1): the oracle against hand-derived cases and invariants,
and the library's host engine against the oracle (bit-exact: both compute the same ratios)."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import step_text as T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "step_text.json")


def _cases():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_oracle_matches_hand_derived_signals(case):
    steps = [tuple(s) for s in case["steps"]]
    for (th, ac, ob), want in zip(steps, case["cues"]):
        assert [c.decode() for c in T.cues(th.encode() + b" " + ob.encode())] == want["th_obs"]
        assert [c.decode() for c in T.cues(ac)] == want["act"]
        assert [c.decode() for c in T.cues(ob)] == want["obs"]
    valid, gain, red, obs_sim = T.step_signals(steps)
    assert valid.tolist() == case["valid"]
    assert gain.tolist() == [float(Fraction(x)) for x in case["gain"]]
    assert red.tolist() == [float(Fraction(x)) for x in case["red"]]
    assert obs_sim.tolist() == [[float(Fraction(x)) for x in row] for row in case["obs_sim"]]


def test_sim_properties():
    a, b, e = T.cues("alpha beta gamma"), T.cues("gamma delta"), T.cues("")
    assert T.sim(a, b) == T.sim(b, a) == 1 / 4
    assert T.sim(a, a) == 1.0 and T.sim(e, e) == 0.0 and T.sim(a, e) == 0.0


def test_cue_rules():
    assert T.cues("The THE the x 7 42 ab") == [b"42", b"ab"]  # stop words, 1-byte runs, case
    words = " ".join(f"k{i:03d}" for i in range(100))
    got = T.cues(words + " k000")
    assert len(got) == T.CUE_CAP and got[0] == b"k000" and got[-1] == b"k063"
    assert T.cues("foo_bar-baz.qux") == [b"foo", b"bar", b"baz", b"qux"]


def test_validity_rules():
    assert T.observation_valid("Found 3 results about Paris.") == 1
    assert T.observation_valid("") == 0 and T.observation_valid("  a ") == 0  # no cue
    for bad in ("Error 404", "  exception raised", "Traceback (most recent call last)",
                "No results for query", "NOT FOUND", "timed out after 30 s"):
        assert T.observation_valid(bad) == 0, bad
    assert T.observation_valid("The error was fixed later") == 1  # a marker inside is fine


# ---------------------------------------------------------------- the library's host engine
def _fnv1a64(data: bytes) -> int:
    """64-bit FNV-1a (the published offset basis and prime)."""
    h = 0xcbf29ce484222325
    for b in data:
        h ^= b
        h = (h * 0x100000001b3) & 0xFFFFFFFFFFFFFFFF
    return h


@pytest.fixture(scope="module")
def B():
    from paper_2609_22158_amd import binding

    binding.load()
    return binding


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_engine_matches_golden(B, case):
    tr = B.TextTracker(len(case["steps"]))
    for t, (th, ac, ob) in enumerate(case["steps"]):
        v, g, r, sim = tr.signals(th, ac, ob)
        assert v == case["valid"][t]
        assert g == np.float32(float(Fraction(case["gain"][t])))
        assert r == np.float32(float(Fraction(case["red"][t])))
        want = [np.float32(float(Fraction(x))) for x in case["obs_sim"][t][:t]]
        assert sim.tolist() == want


@pytest.mark.parametrize("seed", [233, 42, 3407])
def test_engine_cues_match_oracle(B, seed):
    from synth.text import make_text_trajectory

    for th, ac, ob in make_text_trajectory(seed, 30):
        for text in (th, ac, ob, th + " " + ob):
            want = [_fnv1a64(c) for c in T.cues(text)]
            assert B.text_cues(text).tolist() == want, text[:60]


@pytest.mark.parametrize("seed", [233, 42, 3407])
def test_engine_signals_and_utilities_match_oracle(B, seed):
    """Bit-exact signals (both sides take the same ratios in double, cast to float),
    and utilities within float rounding of the oracle's fp64 Algorithm 1."""
    import oracle as O
    from synth.text import make_text_trajectory

    steps = make_text_trajectory(seed, 60)
    valid, gain, red, obs_sim = T.step_signals(steps)
    assert 0 < valid.sum() < len(steps) and red.max() == 1.0 and obs_sim.max() > 0  # all paths
    tr = B.TextTracker(len(steps))
    for t, (th, ac, ob) in enumerate(steps):
        S = tr.update(th, ac, ob)
        _, _, S_o = O.run_step_updates(valid[:t + 1], gain[:t + 1], red[:t + 1],
                                       obs_sim[:t + 1, :t + 1], O.Params())
        np.testing.assert_allclose(S, S_o, rtol=2e-7, atol=2e-7)
    tr2 = B.TextTracker(len(steps))
    for t, (th, ac, ob) in enumerate(steps):
        v, g, r, sim = tr2.signals(th, ac, ob)
        assert (v, g, r) == (np.float32(valid[t]), np.float32(gain[t]), np.float32(red[t])), t
        assert sim.tolist() == obs_sim[t, :t].astype(np.float32).tolist(), t


def test_engine_rejects(B):
    import ctypes

    lib = B.load()
    out = ctypes.c_float()
    p = ctypes.byref(out)
    st = np.zeros(8, np.uint64)  # never initialised
    assert lib.stepkv_text_step(st.ctypes.data, b"", 0, b"", 0, b"", 0, p, p, p, None) == B.EINVAL
    assert lib.stepkv_text_state_bytes(0) == 0
    n = lib.stepkv_text_state_bytes(1)
    st = np.zeros((n + 7) // 8, np.uint64)
    assert lib.stepkv_text_state_init(st.ctypes.data, n - 1, 1) == B.EINVAL
    assert lib.stepkv_text_state_init(st.ctypes.data, n, 1) == 0
    assert lib.stepkv_text_step(st.ctypes.data, None, 3, b"", 0, b"", 0, p, p, p, None) == B.EINVAL
    assert lib.stepkv_text_step(st.ctypes.data, b"a", 1, b"", 0, b"", -1, p, p, p, None) == B.EINVAL
    assert lib.stepkv_text_step(st.ctypes.data, b"a", 1, b"", 0, b"", 0, p, p, p, None) == 0
    sim = (ctypes.c_float * 2)()
    assert lib.stepkv_text_step(st.ctypes.data, b"a", 1, b"", 0, b"", 0, p, p, p, sim) == B.EINVAL  # full
