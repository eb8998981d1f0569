"""Seeded ReAct-shaped trajectory text (Thought, Action, Observation per step)
for the text step-signal engine. The words are made up from syllables; no
benchmark content is used. Holds none of the method's arithmetic."""
from __future__ import annotations

from typing import List, Tuple

import numpy as np

_SYL = ["ka", "ro", "mi", "tel", "van", "dor", "ish", "lu", "pe", "zan", "qui", "bor", "sa",
        "nel", "ti", "gar", "fo", "ren", "cho", "wix"]
_FUNCTION = ["the", "of", "and", "to", "in", "is", "was", "for", "on", "with", "a", "it", "that",
             "by", "from", "this", "not", "but", "also", "which"]
_NON_ASCII = ["café", "naïve", "Zürich", "São", "Kraków", "façade", "résumé", "Ångström"]
_ERRORS = ["Error: the page could not be retrieved.", "  Timeout while contacting the server",
           "No results found for the query.", "Exception: rate limit exceeded", "Not found."]
_TOOLS = ["Search", "Lookup", "Open", "Finish"]


def _vocab(rng, n: int) -> List[str]:
    words = set()
    while len(words) < n:
        k = int(rng.integers(2, 4))
        words.add("".join(rng.choice(_SYL, size=k)))
    return sorted(words)


def make_text_trajectory(seed: int, num_steps: int = 40, vocab: int = 300
                         ) -> List[Tuple[str, str, str]]:
    rng = np.random.default_rng(seed)
    V = _vocab(rng, vocab)
    steps: List[Tuple[str, str, str]] = []

    def words(n):
        out = []
        for _ in range(n):
            r = rng.random()
            if r < 0.30:
                out.append(str(rng.choice(_FUNCTION)))
            elif r < 0.34:
                out.append(str(rng.choice(_NON_ASCII)))
            elif r < 0.40:
                out.append(str(int(rng.integers(0, 3000))))
            else:
                w = str(rng.choice(V))
                out.append(w.capitalize() if rng.random() < 0.2 else w)
        return out

    for t in range(num_steps):
        thought = " ".join(words(int(rng.integers(0, 16)))) + "."
        if t > 0 and rng.random() < 0.25:
            action = steps[int(rng.integers(0, t))][1]  # a repeated tool call
        else:
            action = f"{rng.choice(_TOOLS)}[{' '.join(words(int(rng.integers(1, 4))))}]"
        r = rng.random()
        if r < 0.08:
            obs = str(rng.choice(_ERRORS))
        elif r < 0.12:
            obs = " " * int(rng.integers(0, 3))
        else:
            body = words(int(rng.integers(10, 140)))  # long ones pass the 64-cue cap
            if t > 0 and rng.random() < 0.35:  # part of an earlier observation comes back
                prev = steps[int(rng.integers(0, t))][2].split()
                if prev:
                    a = int(rng.integers(0, len(prev)))
                    body = prev[a:a + int(rng.integers(5, 40))] + body
            obs = " ".join(body)
        steps.append((thought, action, obs))
    return steps
