"""Host code of the library under AddressSanitizer and UndefinedBehaviorSanitizer.

Run by tests/test_host_sanitizers.py in a child process that preloads the
sanitizer runtime and loads the sanitized build (STEPKV_LIB); a sanitizer
report ends that process with its own exit code, which fails the parent test.
Hypothesis draws the inputs: arbitrary byte strings (NUL, non-ASCII, long runs,
the cue cap and beyond) through the text engine, signal values (NaN, inf,
out-of-range similarities) through the step update, and arbitrary problem
descriptors and parameters through the argument validation of every device
entry point. The device calls here always get a NULL required pointer, so
every one of them returns during validation and none reaches a kernel.
Results are checked against the oracle where the oracle defines them.
"""
import ctypes
import math

import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle import step_text as T
import oracle as O
from paper_2609_22158_amd import binding as B

LIB = B.load()
_KEEP = []


def buf(b: bytes):
    """The bytes in a fresh heap block of exactly len(b) bytes (no terminator), so that a
    read past the end lands in the sanitizer's redzone; returned as a char pointer."""
    arr = np.empty(max(len(b), 1), np.uint8)[:len(b)]  # numpy allocates with malloc
    arr = np.frombuffer(b, np.uint8).copy() if b else arr
    _KEEP.append(arr)
    return ctypes.cast(arr.ctypes.data, ctypes.c_char_p)
FAKE = 0x10000  # placeholder device address (every call below fails validation first)
SETTINGS = settings(max_examples=300, deadline=None, derandomize=True,
                    suppress_health_check=list(HealthCheck))

words = st.sampled_from([b"alpha", b"Beta", b"the", b"error", b"not found", b"42", b"x",
                         b"\xc3\xa9t\xc3\xa9", b"\x00", b"   ", b"timeout", b"Paris", b"a1b2"])
# the error markers and every proper prefix of them (a text may end inside a marker)
markers = [b"error", b"exception", b"traceback", b"invalid", b"failed", b"failure",
           b"no results", b"not found", b"timed out", b"timeout"]
near_markers = st.sampled_from([m[:k] for m in markers for k in range(1, len(m) + 1)])
texts = st.one_of(st.binary(max_size=600),
                  st.lists(words, max_size=160).map(lambda ws: b" ".join(ws)),
                  st.tuples(st.sampled_from([b"", b"  ", b"\t\n"]), near_markers,
                            st.booleans()).map(lambda t: t[0] + (t[1].upper() if t[2] else t[1])))


@SETTINGS
@given(st.lists(st.tuples(texts, texts, texts), min_size=1, max_size=12),
       st.integers(min_value=1, max_value=14))
def check_text_engine(steps, capacity):
    nbytes = LIB.stepkv_text_state_bytes(capacity)
    state = np.zeros((nbytes + 7) // 8, np.uint64)
    assert LIB.stepkv_text_state_init(state.ctypes.data, nbytes, capacity) == 0
    v, g, r = ctypes.c_float(), ctypes.c_float(), ctypes.c_float()
    sim = np.zeros(capacity, np.float32)
    out = []
    for t, (th, ac, ob) in enumerate(steps):
        rc = LIB.stepkv_text_step(state.ctypes.data, buf(th), len(th), buf(ac), len(ac),
                                  buf(ob), len(ob),
                                  ctypes.byref(v), ctypes.byref(g), ctypes.byref(r),
                                  sim.ctypes.data_as(B._f32p))
        if t >= capacity:
            assert rc == B.EINVAL  # a full state is refused
            break
        assert rc == 0
        out.append((v.value, g.value, r.value, sim[:t].copy()))
        _KEEP.clear()
    n = len(out)
    valid, gain, red, obs_sim = T.step_signals([tuple(s) for s in steps[:n]])
    for t, (vv, gg, rr, ss) in enumerate(out):
        assert vv == valid[t]
        assert math.isclose(gg, gain[t], rel_tol=0, abs_tol=1e-6)
        assert math.isclose(rr, red[t], rel_tol=0, abs_tol=1e-6)
        np.testing.assert_allclose(ss, obs_sim[t, :t], rtol=0, atol=1e-6)
    # a negative length and a NULL text with a positive length are refused
    fresh = np.zeros_like(state)
    assert LIB.stepkv_text_state_init(fresh.ctypes.data, nbytes, capacity) == 0
    assert LIB.stepkv_text_step(fresh.ctypes.data, b"a", -1, b"", 0, b"", 0, ctypes.byref(v),
                                ctypes.byref(g), ctypes.byref(r), None) == B.EINVAL
    assert LIB.stepkv_text_step(fresh.ctypes.data, None, 3, b"", 0, b"", 0, ctypes.byref(v),
                                ctypes.byref(g), ctypes.byref(r), None) == B.EINVAL


@SETTINGS
@given(texts)
def check_text_cues(text):
    cues = (ctypes.c_uint64 * B.CUE_CAP)()
    n = ctypes.c_int32(-1)
    assert LIB.stepkv_text_cues(buf(text), len(text), cues, ctypes.byref(n)) == 0
    _KEEP.clear()
    assert 0 <= n.value <= B.CUE_CAP
    assert n.value == len(T.cues(text))


signal = st.one_of(st.floats(allow_nan=True, allow_infinity=True, width=32),
                   st.floats(min_value=0, max_value=1, width=32))


@SETTINGS
@given(st.lists(st.tuples(signal, signal, signal,
                          st.lists(st.one_of(signal, st.floats(-2, 3, width=32)),
                                   max_size=20)), min_size=1, max_size=20),
       st.integers(min_value=1, max_value=21))
def check_step_update(boundaries, capacity):
    r = np.zeros(capacity)
    c = np.zeros(capacity)
    stt = B.StepStateC(capacity, 0, r.ctypes.data_as(B._f64p), c.ctypes.data_as(B._f64p))
    prm = B.Params().c()
    S = np.zeros(capacity, np.float32)
    for valid, gain, red, sims in boundaries:
        t = stt.num_steps
        sim = np.zeros(max(t, 1), np.float32)
        sim[:min(t, len(sims))] = sims[:t]
        rc = LIB.stepkv_step_update(ctypes.byref(stt), valid, gain, red,
                                    sim.ctypes.data_as(B._f32p), ctypes.byref(prm),
                                    S.ctypes.data_as(B._f32p))
        ok = (t < capacity and all(math.isfinite(x) for x in (valid, gain, red))
              and all(0.0 <= float(x) <= 1.0 for x in sim[:t]))
        assert (rc == 0) == ok, (rc, t, capacity)
        if rc == 0:
            assert stt.num_steps == t + 1 and np.all((S[:t + 1] >= 0) & (S[:t + 1] <= 8))
    assert LIB.stepkv_step_update(None, 1.0, 1.0, 0.0, None, ctypes.byref(prm),
                                  S.ctypes.data_as(B._f32p)) == B.EINVAL


problems = st.fixed_dictionaries({
    "L": st.integers(-2, 70), "Hq": st.integers(-1, 70), "Hkv": st.integers(-1, 9),
    "d": st.sampled_from([0, 64, 96, 128, 256, -64]), "W": st.integers(-1, 300),
    "lens": st.lists(st.integers(-5, 40000), min_size=1, max_size=20),
    "steps": st.lists(st.integers(-2, 5000), min_size=1, max_size=20),
})


def _problem(p):
    S = len(p["lens"])
    cu = np.concatenate([[0], np.cumsum(p["lens"])]).astype(np.int64)
    cu = np.clip(cu, -2**31, 2**31 - 1).astype(np.int32)
    steps = (p["steps"] * S)[:S]
    cs = np.clip(np.concatenate([[0], np.cumsum(steps)]), -2**31, 2**31 - 1).astype(np.int32)
    pb = B.ProblemC(p["L"], p["Hq"], p["Hkv"], p["d"], p["W"], S, cu.ctypes.data_as(B._i32p),
                    FAKE, cs.ctypes.data_as(B._i32p), FAKE, None)
    return pb, cu, cs


params = st.builds(lambda a, b, k, sc, ct: B.Params(alpha=a, beta=b, pool_kernel=k, scale=sc,
                                                    causal_tail=ct).c(),
                   st.floats(width=32), st.floats(width=32), st.integers(-3, 70),
                   st.floats(width=32), st.integers(0, 1))


@SETTINGS
@given(problems, params, st.integers(-5, 5000))
def check_device_call_validation(p, prm, budget):
    pb, cu, cs = _problem(p)
    P, R = ctypes.byref(pb), ctypes.byref(prm)
    for fn in ("stepkv_score_workspace_bytes", "stepkv_saliency_workspace_bytes",
               "stepkv_compress_workspace_bytes"):
        getattr(LIB, fn)(P)
    LIB.stepkv_score_shared_workspace_bytes(P, 3)
    LIB.stepkv_decode_workspace_bytes(P, max(budget, 0))
    big = 1 << 40
    # every device call gets a NULL required pointer: validation returns before any launch
    assert LIB.stepkv_score(P, R, None, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, FAKE * 16,
                            big, None) < 0
    assert LIB.stepkv_score_noalloc(P, R, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                    None) < 0
    assert LIB.stepkv_saliency(P, R, FAKE, None, FAKE, FAKE * 16, big, None) < 0
    assert LIB.stepkv_priority(P, R, None, FAKE, FAKE, FAKE, FAKE, None, None) < 0
    assert LIB.stepkv_select(P, None, FAKE, FAKE, budget, None, FAKE, FAKE, None, None) < 0
    assert LIB.stepkv_compact(P, FAKE, None, FAKE, FAKE, budget, FAKE, FAKE, None) < 0
    assert LIB.stepkv_compress(P, R, FAKE, FAKE, None, None, FAKE, FAKE, FAKE, budget, None,
                               None, None, FAKE, max(budget, 0), FAKE, FAKE, FAKE * 16, big,
                               None) < 0
    assert LIB.stepkv_decode_attention(P, None, FAKE, FAKE, FAKE, max(budget, 0), 0.0, FAKE,
                                       FAKE * 16, big, None) < 0
    assert LIB.stepkv_score_shared(P, R, None, FAKE, None, 3, FAKE, FAKE, FAKE, FAKE, None,
                                   None, FAKE * 16, big, None) < 0
    # the host retained-row rule on the same descriptor and a drawn mask
    ntot = int(cu[-1]) if (np.diff(cu) >= 0).all() and cu[-1] >= 0 else 0
    prot = (np.arange(max(ntot, 1)) % 7 == 0).astype(np.uint8)
    out = np.zeros(len(cu), np.int32)
    rc = LIB.stepkv_retained_rows(P, prot.ctypes.data, budget, None, out.ctypes.data)
    valid = (np.diff(cu) >= 0).all() and cu[0] == 0 and budget >= 1 and pb.num_seqs >= 1
    assert (rc == 0) == bool(valid)
    if rc == 0:
        want = [0]
        for s in range(pb.num_seqs):
            n = int(cu[s + 1] - cu[s])
            np_ = int(prot[cu[s]:cu[s + 1]].sum())
            want.append(want[-1] + O.retained_count(n, np_, budget))
        assert out.tolist() == want


def main():
    for case in (check_text_cues, check_text_engine, check_step_update,
                 check_device_call_validation):
        case()
        print(f"{case.__name__}: ok", flush=True)


if __name__ == "__main__":
    main()
