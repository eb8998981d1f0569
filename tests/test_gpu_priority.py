"""stepkv_priority without step statistics, where every (layer, KV head) row is spread over
workgroups of 2048 positions (three launches; the chunk maxima wait in the scores row): here
8 layers x 4 KV heads x 9 sequences = 288 rows, more than the 256 up to which the
per-sequence kernel is kept.

Against the per-sequence kernels that also gather the step statistics (the call with
step_stats): bit for bit, since both pool the window left to right from its first position,
take the same maximum and fuse with the same operations. Against the oracle's eq.
token-priority (pooled_saliency, normalised_saliency, priority) within the parity tolerance.

Inputs: seeded saliency rows (exponential values, exact zeros, one all-zero row so that the
maximum is 0), protected prefixes plus scattered protected tokens, step ids with some out of
range, sequence lengths on both sides of the 2048-position chunks and past the 32768 that
the register path of the per-sequence kernel holds, pooling windows 1 to 63.
"""
import numpy as np
import pytest

import oracle as O
from tests.gpu_cases import close, log

pytestmark = pytest.mark.gpu

SEQLENS = [1, 2047, 2048, 2049, 5000, 0, 4096, 40000, 3]


def _inputs(seed, L=8, Hkv=4):
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(SEQLENS)]).astype(np.int32)
    ntot = int(cu[-1])
    nsteps = [max(1, n // 400) for n in SEQLENS]
    cu_steps = np.concatenate([[0], np.cumsum(nsteps)]).astype(np.int32)
    sal = rng.exponential(1.0, (L, Hkv, ntot)).astype(np.float32)
    sal[rng.random((L, Hkv, ntot)) < 0.05] = 0.0
    sal[1, 1] = 0.0  # a row whose maximum is 0: Th = 0 everywhere
    prot = (rng.random(ntot) < 0.1).astype(np.uint8)
    sid = np.empty(ntot, np.int32)
    for s, n in enumerate(SEQLENS):
        a, b = int(cu[s]), int(cu[s + 1])
        prot[a:a + min(n, 64)] = 1
        ids = np.sort(rng.integers(0, nsteps[s], n)).astype(np.int32)
        bad = rng.random(n) < 0.01
        ids[bad] = rng.choice(np.array([-1, nsteps[s], 1 << 20], np.int32), int(bad.sum()))
        sid[a:b] = ids
    util = rng.random(int(cu_steps[-1])).astype(np.float32)
    return cu, cu_steps, sal, prot, sid, util


@pytest.mark.parametrize("pool", [1, 7, 9, 15, 63])
def test_row_spread_priority_matches_per_sequence_kernels_and_oracle(pool):
    import torch

    from paper_2609_22158_amd import binding as B

    cu, cu_steps, sal, prot, sid, util = _inputs(1000 + pool)
    L, Hkv = sal.shape[:2]
    pb = B.Problem(L, 4 * Hkv, Hkv, 128, 32, cu, cu_steps, status=False)
    prm = B.Params(alpha=0.3, beta=0.7, pool_kernel=pool)
    args = [torch.from_numpy(x).cuda() for x in (sal, sid, prot, util)]
    log(f"[priority pool {pool}] seqlens={SEQLENS}")
    spread = B.priority(pb, *args, prm)["scores"].cpu().numpy()
    per_seq = B.priority(pb, *args, prm, want_stats=True)["scores"].cpu().numpy()
    assert np.array_equal(spread.view(np.uint32), per_seq.view(np.uint32))
    for s, n in enumerate(SEQLENS):
        a, b = int(cu[s]), int(cu[s + 1])
        prun = prot[a:b] == 0
        S = util[int(cu_steps[s]):int(cu_steps[s + 1])].astype(np.float64)
        for l in range(L):
            for h in range(Hkv):
                T = O.pooled_saliency(sal[l, h, a:b].astype(np.float64), prun, pool)
                ref = O.priority(O.normalised_saliency(T, prun), sid[a:b], S, prun, 0.3, 0.7)
                close(spread[l, h, a:b], ref, f"P{(s, l, h)} pool {pool}")


def test_row_spread_priority_reports_conditions():
    """The row-spread path's checked variant (a status word in the problem): the inputs above
    hold prunable tokens with out-of-range step ids (STEPKV_FLAG_STEP_ID); a NaN saliency adds
    STEPKV_FLAG_NONFINITE; with every step id in range and finite inputs nothing is reported.
    The scores are the unchecked variant's in every case."""
    import torch

    from paper_2609_22158_amd import binding as B

    cu, cu_steps, sal, prot, sid, util = _inputs(77)
    L, Hkv = sal.shape[:2]
    pb = B.Problem(L, 4 * Hkv, Hkv, 128, 32, cu, cu_steps, status=True)
    quiet = B.Problem(L, 4 * Hkv, Hkv, 128, 32, cu, cu_steps, status=False)
    prm = B.Params(pool_kernel=7)
    clean_sid = sid.copy()
    for s in range(len(SEQLENS)):
        a, b = int(cu[s]), int(cu[s + 1])
        n = int(cu_steps[s + 1] - cu_steps[s])
        clean_sid[a:b] = np.clip(sid[a:b], 0, n - 1)
    nan_sal = sal.copy()
    nan_sal[3, 2, int(cu[7]) + 12345] = np.nan  # a prunable position of the 40000-token sequence
    prot_n = prot.copy()
    prot_n[int(cu[7]) + 12345] = 0
    cases = [("bad step ids", sal, sid, prot, B.FLAG_STEP_ID),
             ("clean", sal, clean_sid, prot, 0),
             ("NaN saliency", nan_sal, clean_sid, prot_n, B.FLAG_NONFINITE),
             ("both", nan_sal, sid, prot_n, B.FLAG_STEP_ID | B.FLAG_NONFINITE)]
    pb.status(clear=True)
    for what, a_, s_, p_, want in cases:
        args = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in (a_, s_, p_, util)]
        log(f"[priority flags] {what}")
        checked = B.priority(pb, *args, prm)["scores"].cpu().numpy()
        assert pb.status(clear=True) == want, what
        plain = B.priority(quiet, *args, prm)["scores"].cpu().numpy()
        assert np.array_equal(checked.view(np.uint32), plain.view(np.uint32)), what


def test_many_steps_take_the_spread_path_against_oracle():
    """More than 4096 steps in a sequence (here 5000 steps of 2-3 tokens): the per-sequence
    kernels would stage every step utility in LDS, so the row-spread path runs even for three
    rows (a row count that leaves the last group of rows per workgroup partly empty), reading
    the utilities from memory. Against the oracle's eq. token-priority."""
    import torch

    from paper_2609_22158_amd import binding as B

    rng = np.random.default_rng(4242)
    n, nsteps = 12345, 5000
    cu = np.array([0, n], np.int32)
    cu_steps = np.array([0, nsteps], np.int32)
    sal = rng.exponential(1.0, (1, 3, n)).astype(np.float32)
    prot = np.zeros(n, np.uint8)
    prot[:100] = 1
    sid = np.minimum(np.arange(n) * nsteps // n, nsteps - 1).astype(np.int32)
    util = rng.random(nsteps).astype(np.float32)
    pb = B.Problem(1, 12, 3, 128, 32, cu, cu_steps, status=False)
    prm = B.Params(alpha=0.4, beta=0.6, pool_kernel=7)
    log("[priority] 5000 steps in one sequence")
    got = B.priority(pb, *[torch.from_numpy(x).cuda() for x in (sal, sid, prot, util)],
                     prm)["scores"].cpu().numpy()
    prun = prot == 0
    for h in range(3):
        T = O.pooled_saliency(sal[0, h].astype(np.float64), prun, 7)
        ref = O.priority(O.normalised_saliency(T, prun), sid, util.astype(np.float64), prun, 0.4, 0.6)
        close(got[0, h], ref, f"P head {h}")
