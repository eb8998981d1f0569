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
