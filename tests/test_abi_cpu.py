"""C ABI checks that need no GPU: exports, host helpers and argument validation.

Validation runs on the host before any HIP call, so the device pointers below
are never dereferenced (they are placeholders).
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
from paper_2609_22158_amd import binding as B
from synth import make_workload

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "stepkv.h")
FAKE = 0x10000  # placeholder device address; never dereferenced by these calls
FAR = 1 << 44  # another placeholder, far enough from FAKE that no array here spans both


@pytest.fixture(scope="module")
def lib():
    return B.load()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(stepkv_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_function(lib):
    names = _declared_functions()
    assert len(names) == 31, names
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B._SIGNATURES)


def test_defaults_are_the_papers(lib):
    p = B.Params.library_default()
    assert (round(p.alpha, 6), round(p.beta, 6)) == (0.2, 0.8)
    assert (round(p.lambda_red, 6), round(p.w_r, 6), round(p.w_c, 6)) == (0.3, 0.85, 0.15)
    assert (p.r_min, p.r_max, p.s_max, p.eta, p.pool_kernel) == (-1.0, 2.0, 8.0, 1.5, 7)
    assert p.causal_tail == 0  # every window row sees the whole sequence unless asked


def test_strerror(lib):
    assert B.strerror(0) == "ok"
    assert "workspace" in B.strerror(-3)


@pytest.mark.parametrize("rho,n", [(0.2, 1000), (0.2, 3), (0.29, 100), (0.5, 7), (1.0, 9), (0.3, 0)])
def test_budget_from_ratio_matches_oracle(lib, rho, n):
    assert B.budget_from_ratio(rho, n) == O.budget_from_ratio(rho, n)


def test_budget_from_ratio_rejects(lib):
    assert B.budget_from_ratio(0.0, 10) == -1
    assert B.budget_from_ratio(1.5, 10) == -1
    assert B.budget_from_ratio(0.5, -1) == -1


@pytest.mark.parametrize("seed", [233, 42, 3407])
def test_host_step_update_matches_oracle(lib, seed):
    w = make_workload("l32_32k", seed, num_layers=1, with_v=False)
    sig = w.signals[0]
    S_c = B.step_utilities(sig.valid, sig.gain, sig.red, sig.obs_sim)
    _, c_o, S_o = O.run_step_updates(sig.valid, sig.gain, sig.red,
                                     sig.obs_sim.astype(np.float64), O.Params())
    np.testing.assert_allclose(S_c, S_o, rtol=2e-7, atol=2e-7)
    # planted steps are reused at every later boundary: min(1, 1.5 * sim) >= 0.75 each time
    n = sig.num_steps
    for k in w.planted_steps[0]:
        assert c_o[k] >= 0.75 * (n - 1 - k) - 1e-9


def test_host_step_update_rejects(lib):
    p = B.Params().c()
    r = np.zeros(2)
    c = np.zeros(2)
    st = B.StepStateC(2, 0, r.ctypes.data_as(B._f64p), c.ctypes.data_as(B._f64p))
    S = np.zeros(2, np.float32)
    Sp = S.ctypes.data_as(B._f32p)
    assert lib.stepkv_step_update(ctypes.byref(st), 1, 1, 0, None, ctypes.byref(p), Sp) == 0
    bad = np.array([1.5], np.float32)
    assert lib.stepkv_step_update(ctypes.byref(st), 1, 1, 0, bad.ctypes.data_as(B._f32p),
                                  ctypes.byref(p), Sp) == B.EINVAL
    assert lib.stepkv_step_update(ctypes.byref(st), 1, 1, 0, None, ctypes.byref(p), Sp) == B.EINVAL
    ok = np.array([0.5], np.float32)
    assert lib.stepkv_step_update(ctypes.byref(st), 1, 0.5, 0, ok.ctypes.data_as(B._f32p),
                                  ctypes.byref(p), Sp) == 0
    assert lib.stepkv_step_update(ctypes.byref(st), 1, 1, 0, ok.ctypes.data_as(B._f32p),
                                  ctypes.byref(p), Sp) == B.EINVAL  # capacity 2 reached
    assert S[0] == pytest.approx(0.85 * 2 + 0.15 * np.log(1.75), abs=1e-6)


def _problem(L=2, Hq=8, Hkv=2, d=128, W=32, cu=(0, 1000, 3000), cu_steps=(0, 4, 9)):
    cu = np.array(cu, np.int32)
    cs = np.array(cu_steps, np.int32)
    pb = B.ProblemC(L, Hq, Hkv, d, W, len(cu) - 1, cu.ctypes.data_as(B._i32p), FAKE,
                    cs.ctypes.data_as(B._i32p), FAKE)
    pb._keep = (cu, cs)
    return pb


def _score(lib, pb, prm=None, ws_bytes=None, **ptrs):
    prm = prm or B.Params().c()
    args = dict(q=FAKE, k=FAKE, sid=FAKE, prot=FAKE, util=FAKE, scores=FAKE, sal=None, stats=None,
                ws=FAKE * 16)
    args.update(ptrs)
    need = lib.stepkv_score_workspace_bytes(ctypes.byref(pb))
    return lib.stepkv_score(ctypes.byref(pb), ctypes.byref(prm), args["q"], args["k"], args["sid"],
                            args["prot"], args["util"], args["scores"], args["sal"],
                            args["stats"], args["ws"], need if ws_bytes is None else ws_bytes,
                            None)


def test_workspace_bytes(lib):
    pb = _problem()
    n = lib.stepkv_score_workspace_bytes(ctypes.byref(pb))
    # at least the fp32 saliency of every (layer, head, token)
    assert n >= 4 * 2 * 2 * 3000 and n % 256 == 0
    assert lib.stepkv_score_workspace_bytes(ctypes.byref(_problem(Hq=7))) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(Hq=7), B.EINVAL),          # G not an integer
    (dict(d=96), B.EUNSUPPORTED),    # head dim
    (dict(d=0), B.EINVAL),
    (dict(W=513, Hq=8, Hkv=2), B.EUNSUPPORTED),  # W*G = 2052 > 2048
    (dict(cu=(0, 10, 5)), B.EINVAL),  # not monotone
    (dict(cu=(1, 10, 20)), B.EINVAL),  # does not start at 0
    (dict(L=0), B.EINVAL),
])
def test_score_rejects_problem(lib, kw, code):
    assert _score(lib, _problem(**kw)) == code


def test_score_rejects_arguments(lib):
    pb = _problem()
    assert _score(lib, pb, q=None) == B.EINVAL
    assert _score(lib, pb, scores=None) == B.EINVAL
    assert _score(lib, pb, util=None) == B.EINVAL
    assert _score(lib, pb, ws=None) == B.EWORKSPACE
    assert _score(lib, pb, ws_bytes=1024) == B.EWORKSPACE
    assert _score(lib, pb, ws=FAKE * 16 + 8) == B.EWORKSPACE  # misaligned
    assert _score(lib, pb, prm=B.Params(pool_kernel=6).c()) == B.EINVAL
    assert _score(lib, pb, prm=B.Params(pool_kernel=65).c()) == B.EUNSUPPORTED
    assert _score(lib, pb, prm=B.Params(saliency_schedule=3).c()) == B.EINVAL
    assert _score(lib, pb, prm=B.Params(saliency_schedule=-1).c()) == B.EINVAL
    assert _score(lib, pb, prm=B.Params(alpha=float("nan")).c()) == B.EINVAL
    many = _problem(cu_steps=(0, 4097, 4099))
    assert _score(lib, many, stats=FAKE) == B.EUNSUPPORTED


def test_saliency_priority_reject(lib):
    pb = _problem()
    prm = B.Params().c()
    need = lib.stepkv_saliency_workspace_bytes(ctypes.byref(pb))
    assert 0 < need < lib.stepkv_score_workspace_bytes(ctypes.byref(pb))
    sal = lib.stepkv_saliency
    assert sal(ctypes.byref(pb), ctypes.byref(prm), FAKE, FAKE, None, FAKE * 16, need,
               None) == B.EINVAL
    assert sal(ctypes.byref(pb), ctypes.byref(prm), FAKE, FAKE, FAKE, FAKE * 16, need - 256,
               None) == B.EWORKSPACE
    assert sal(ctypes.byref(_problem(W=513)), ctypes.byref(prm), FAKE, FAKE, FAKE, FAKE * 16,
               need, None) == B.EUNSUPPORTED
    pri = lib.stepkv_priority
    assert pri(ctypes.byref(pb), ctypes.byref(prm), None, FAKE, FAKE, FAKE, FAKE, None,
               None) == B.EINVAL
    # saliency and scores sharing memory (the row-spread priority keeps partial maxima in
    # the scores rows while other workgroups still read the saliency around them)
    n = 2 * 2 * 3000 * 4  # L * Hkv * Ntot floats
    assert pri(ctypes.byref(pb), ctypes.byref(prm), FAKE, FAKE, FAKE, FAKE, FAKE, None,
               None) == B.EINVAL
    assert pri(ctypes.byref(pb), ctypes.byref(prm), FAKE + n - 4, FAKE, FAKE, FAKE, FAKE, None,
               None) == B.EINVAL
    assert pri(ctypes.byref(pb), ctypes.byref(B.Params(pool_kernel=0).c()), FAKE, FAKE, FAKE,
               FAKE, FAKE, None, None) == B.EINVAL


def test_select_compact_decode_reject(lib):
    pb = _problem()
    assert lib.stepkv_select(ctypes.byref(pb), FAKE, FAKE, FAKE, 0, None, FAKE, FAKE, None,
                             None) == B.EINVAL  # budget < 1
    assert lib.stepkv_select(ctypes.byref(pb), None, FAKE, FAKE, 4, None, FAKE, FAKE, None,
                             None) == B.EINVAL
    assert lib.stepkv_select(ctypes.byref(pb), FAKE, FAKE, None, 4, None, FAKE, FAKE, FAKE,
                             None) == B.EINVAL  # kept needs step ids
    assert lib.stepkv_compact(ctypes.byref(pb), FAKE, FAKE, FAKE, FAKE, -1, FAKE, FAKE,
                              None) == B.EINVAL
    assert lib.stepkv_compact(ctypes.byref(pb), FAKE, None, FAKE, FAKE, 8, FAKE, FAKE,
                              None) == B.EINVAL
    assert lib.stepkv_decode_attention(ctypes.byref(_problem(d=80)), FAKE, FAKE, FAKE, FAKE, 8,
                                       0.0, FAKE, FAKE * 16, 1 << 20, None) == B.EUNSUPPORTED
    need = lib.stepkv_decode_workspace_bytes(ctypes.byref(pb), 8)
    assert need > 0
    assert lib.stepkv_decode_attention(ctypes.byref(pb), FAKE, FAKE, FAKE, FAKE, 8, 0.0, FAKE,
                                       FAKE * 16, need - 1, None) == B.EWORKSPACE
    assert lib.stepkv_decode_attention(ctypes.byref(pb), FAKE, FAKE, FAKE, FAKE, 8, 0.0, None,
                                       FAKE * 16, need, None) == B.EINVAL
    assert lib.stepkv_decode_attention(ctypes.byref(pb), FAKE, FAKE, FAKE, FAKE, 8,
                                       float("inf"), FAKE, FAKE * 16, 1 << 20, None) == B.EINVAL


def test_decode_workspace_counts_splits(lib):
    """The decode workspace holds one fp32 state (o[d], m, z) per (layer, KV head, split, head
    of the group); splits of 512 rows number min(sum_s ceil(min(N_s, out_rows) / 512),
    floor(out_rows / 512) + S), the two bounds of sum_s ceil(R_s / 512) the host knows.
    Splits are of 1024 rows instead once L * Hkv * floor(out_rows / 1024) >= 1536."""
    per_split = 2 * 2 * 4 * (128 + 2) * 4  # L * Hkv * G * (d + 2) floats
    for cu, out_rows, splits in [((0, 1000, 3000), 8, 2), ((0, 1000, 3000), 3000, 6),
                                 ((0, 20000, 40000), 1026, 4), ((0, 20000, 40000), 1024, 4),
                                 ((0, 20000, 40000), 1023, 3),
                                 ((0, 400000, 800000), 393215, 769),  # 4 * 383 < 1536
                                 ((0, 400000, 800000), 400000, 392)]:  # 4 * 390: 1024 rows
        pb = _problem(cu=cu)
        assert lib.stepkv_decode_workspace_bytes(ctypes.byref(pb), out_rows) == splits * per_split


def test_lse_entry_points_reject(lib):
    """Validation of the LSE-fed calls: null arguments and short workspaces launch nothing."""
    pb = _problem()
    prm = B.Params().c()
    need = lib.stepkv_saliency_workspace_bytes(ctypes.byref(pb))
    P, R = ctypes.byref(pb), ctypes.byref(prm)
    assert lib.stepkv_window_lse(P, R, FAKE, FAKE, None, FAKE * 16, need, None) == B.EINVAL
    assert lib.stepkv_window_lse(P, R, FAKE, FAKE, FAKE, FAKE * 16, need - 256, None) == B.EWORKSPACE
    assert lib.stepkv_window_lse(P, None, FAKE, FAKE, FAKE, FAKE * 16, need, None) == B.EINVAL
    assert lib.stepkv_saliency_from_lse(P, R, FAKE, FAKE, None, FAKE, FAKE * 16, need,
                                        None) == B.EINVAL
    assert lib.stepkv_saliency_from_lse(P, R, FAKE, FAKE, FAKE, FAKE, FAKE * 16 + 8, need,
                                        None) == B.EWORKSPACE  # misaligned
    full = lib.stepkv_score_workspace_bytes(ctypes.byref(pb))
    args = [FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, FAKE * 16]
    assert lib.stepkv_score_from_lse(P, R, *args, full - 256, None) == B.EWORKSPACE
    args[2] = None  # lse
    assert lib.stepkv_score_from_lse(P, R, *args, full, None) == B.EINVAL
    bad = _problem(W=513)
    assert lib.stepkv_saliency_from_lse(ctypes.byref(bad), R, FAKE, FAKE, FAKE, FAKE, FAKE * 16,
                                        need, None) == B.EUNSUPPORTED


def test_step_tracker_incremental_matches_oracle(lib):
    """Boundary-by-boundary updates (with a snapshot and restore in between) give the
    oracle's utilities after every boundary."""
    w = make_workload("l32_32k", 42, num_layers=1, with_v=False)
    sig = w.signals[0]
    n = sig.num_steps
    tr = B.StepTracker(n)
    snap = None
    for t in range(n):
        if t == n - 1:
            snap = tr.snapshot()
        S = tr.update(sig.valid[t], sig.gain[t], sig.red[t], sig.obs_sim[t, :t])
        _, _, S_o = O.run_step_updates(sig.valid[:t + 1], sig.gain[:t + 1], sig.red[:t + 1],
                                       sig.obs_sim[:t + 1, :t + 1].astype(np.float64), O.Params())
        np.testing.assert_allclose(S, S_o, rtol=2e-7, atol=2e-7)
    out = np.zeros(n, np.float32)
    tr.restore(snap)
    tr.update(sig.valid[n - 1], sig.gain[n - 1], sig.red[n - 1], sig.obs_sim[n - 1, :n - 1], out=out)
    np.testing.assert_array_equal(out, S)
    with pytest.raises(ValueError):
        tr.update(1.0, 0.5, 0.0, np.zeros(3))  # wrong sim_prev length


# ---------------------------------------------------------------- retained rows, compress, status
@pytest.mark.parametrize("seed", range(5))
def test_retained_rows_matches_oracle(lib, seed):
    """stepkv_retained_rows gives the oracle's R_s = P_s + min(B_s, N_s - P_s), prefix-summed,
    for any protected mask (not only a prefix), with one budget or per-sequence budgets
    (below 1 taken as 1, as stepkv_select does)."""
    rng = np.random.default_rng(seed)
    S = int(rng.integers(1, 7))
    lens = rng.integers(0, 300, S)
    lens[rng.integers(0, S)] = 0  # an empty sequence
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    prot = (rng.random(int(cu[-1])) < 0.2).astype(np.uint8)
    pb = _problem(cu=tuple(cu), cu_steps=tuple(np.arange(S + 1)))
    budget = int(rng.integers(1, 200))
    got = np.zeros(S + 1, np.int32)
    assert lib.stepkv_retained_rows(ctypes.byref(pb), prot.ctypes.data, budget, None,
                                    got.ctypes.data) == B.OK
    n_prot = [int(prot[cu[s]:cu[s + 1]].sum()) for s in range(S)]
    want = np.concatenate([[0], np.cumsum([O.retained_count(int(lens[s]), n_prot[s], budget)
                                           for s in range(S)])])
    np.testing.assert_array_equal(got, want)
    budgets = rng.integers(-3, 200, S).astype(np.int32)
    assert lib.stepkv_retained_rows(ctypes.byref(pb), prot.ctypes.data, 0, budgets.ctypes.data,
                                    got.ctypes.data) == B.OK
    want = np.concatenate([[0], np.cumsum([O.retained_count(int(lens[s]), n_prot[s],
                                                            max(1, int(budgets[s])))
                                           for s in range(S)])])
    np.testing.assert_array_equal(got, want)


def test_retained_rows_rejects(lib):
    pb = _problem()
    prot = np.zeros(3000, np.uint8)
    out = np.zeros(3, np.int32)
    f = lib.stepkv_retained_rows
    assert f(None, prot.ctypes.data, 4, None, out.ctypes.data) == B.EINVAL
    assert f(ctypes.byref(pb), None, 4, None, out.ctypes.data) == B.EINVAL
    assert f(ctypes.byref(pb), prot.ctypes.data, 4, None, None) == B.EINVAL
    assert f(ctypes.byref(pb), prot.ctypes.data, 0, None, out.ctypes.data) == B.EINVAL
    assert f(ctypes.byref(_problem(cu=(0, 10, 5))), prot.ctypes.data, 4, None,
             out.ctypes.data) == B.EINVAL
    assert f(ctypes.byref(pb), prot.ctypes.data, 4, None, out.ctypes.data) == B.OK
    assert list(out) == [0, 4, 8]


def _compress(lib, pb, ws_bytes=None, **kw):
    args = dict(prm=B.Params().c(), q=FAKE, k=FAKE, v=FAKE, lse=None, sid=FAKE, prot=FAKE,
                util=FAKE, budget=4, budgets=None, scores=None, idx=None, cu_ret=FAKE,
                out_rows=8, k_out=FAKE, v_out=FAKE, ws=FAKE * 16)
    args.update(kw)
    need = lib.stepkv_compress_workspace_bytes(ctypes.byref(pb))
    a = args
    return lib.stepkv_compress(ctypes.byref(pb), ctypes.byref(a["prm"]), a["q"], a["k"], a["v"],
                               a["lse"], a["sid"], a["prot"], a["util"], a["budget"],
                               a["budgets"], a["scores"], a["idx"], a["cu_ret"], a["out_rows"],
                               a["k_out"], a["v_out"], a["ws"],
                               need if ws_bytes is None else ws_bytes, None)


def test_compress_workspace_and_rejects(lib):
    """stepkv_compress validates the arguments of all three steps before launching any."""
    pb = _problem()
    need = lib.stepkv_compress_workspace_bytes(ctypes.byref(pb))
    score_ws = lib.stepkv_score_workspace_bytes(ctypes.byref(pb))
    # the score workspace plus fp32 scores and int32 positions for every entry
    assert need >= score_ws + 2 * 4 * 2 * 2 * 3000 and need % 256 == 0
    assert lib.stepkv_compress_workspace_bytes(ctypes.byref(_problem(Hq=7))) == 0
    for kw in (dict(q=None), dict(k=None), dict(v=None), dict(sid=None), dict(prot=None),
               dict(util=None), dict(cu_ret=None), dict(k_out=None), dict(v_out=None),
               dict(out_rows=-1), dict(budget=0), dict(prm=B.Params(pool_kernel=4).c())):
        assert _compress(lib, pb, **kw) == B.EINVAL, kw
    assert _compress(lib, pb, ws=None) == B.EWORKSPACE
    assert _compress(lib, pb, ws_bytes=need - 256) == B.EWORKSPACE
    assert _compress(lib, pb, ws=FAKE * 16 + 4) == B.EWORKSPACE
    assert _compress(lib, _problem(d=96)) == B.EUNSUPPORTED
    assert _compress(lib, _problem(W=513)) == B.EUNSUPPORTED


def test_status_read_rejects(lib):
    pb = _problem()  # no status word
    flags = ctypes.c_uint32(0)
    assert lib.stepkv_status_read(ctypes.byref(pb), ctypes.byref(flags), 0, None) == B.EINVAL
    pb.status = FAKE
    assert lib.stepkv_status_read(ctypes.byref(pb), None, 0, None) == B.EINVAL
    assert lib.stepkv_status_read(None, ctypes.byref(flags), 0, None) == B.EINVAL


def test_score_noalloc_rejects(lib):
    """The scratch-only scoring validates like stepkv_score, needs the saliency buffer, and
    refuses a problem whose sweep workspace exceeds the static scratch before launching."""
    prm = B.Params().c()

    def call(pb, p=prm, **kw):
        a = dict(q=FAKE, k=FAKE, sid=FAKE, prot=FAKE, util=FAKE, scores=FAKE, sal=FAR,
                 stats=None)
        a.update(kw)
        return lib.stepkv_score_noalloc(ctypes.byref(pb), ctypes.byref(p) if p else None,
                                        a["q"], a["k"], a["sid"], a["prot"], a["util"],
                                        a["scores"], a["sal"], a["stats"], None)

    pb = _problem()
    assert call(pb, sal=None) == B.EINVAL  # the saliency buffer is required here
    assert call(pb, sal=FAKE + 4) == B.EINVAL  # saliency overlapping the scores
    assert call(pb, p=None) == B.EINVAL
    assert call(pb, q=None) == B.EINVAL
    assert call(pb, scores=None) == B.EINVAL
    assert call(_problem(d=96)) == B.EUNSUPPORTED
    # 64 layers x 8 heads x 256 window rows over 64 sequences of 20000 tokens: the per-chunk
    # partials alone exceed the static scratch
    big = _problem(L=64, Hq=32, Hkv=8, W=64, cu=tuple(range(0, 64 * 20000 + 1, 20000)),
                   cu_steps=tuple(range(65)))
    assert lib.stepkv_saliency_workspace_bytes(ctypes.byref(big)) > B.STATIC_SCRATCH_BYTES
    assert call(big) == B.ESCRATCH
    assert "static scratch" in B.strerror(B.ESCRATCH)


def test_issue_probe_rejects(lib):
    f = lib.stepkv_issue_probe
    assert f(2, 512, 10, FAKE, None) == B.EINVAL
    assert f(-1, 512, 10, FAKE, None) == B.EINVAL
    assert f(0, 0, 10, FAKE, None) == B.EINVAL
    assert f(1, 512, 0, FAKE, None) == B.EINVAL
    assert f(1, 512, 10, None, None) == B.EINVAL


def test_bandwidth_probe_rejects(lib):
    f = lib.stepkv_bandwidth_probe
    assert f(None, FAKE, 1 << 20, 0, None) == B.EINVAL
    assert f(FAKE, None, 1 << 20, 1, None) == B.EINVAL
    assert f(FAKE, FAKE, 0, 0, None) == B.EINVAL
    assert f(FAKE, FAKE, (1 << 20) + 8, 0, None) == B.EINVAL
    assert f(FAKE + 8, FAKE, 1 << 20, 0, None) == B.EINVAL
