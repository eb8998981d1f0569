"""Full-size parity: the 32-layer caches and the ragged 16-sequence batch at their real
sizes, in the launch configuration the bench times, against the oracle.

Scores and saliency within 2e-3 relative (+1e-7 of the head's max); selection bit-exact
when both sides rank the oracle's priorities cast to fp32 (end to end, retained sets may
differ only by tokens tied with the threshold within that tolerance); compaction
bit-exact; decode over the compacted cache within 2e-3 of each output row's largest
magnitude. Heads the oracle does not recompute are checked by invariants.
"""
import numpy as np
import pytest

import oracle as O
from synth import make_workload
from tests.gpu_cases import HipRun, close, log, ref_rows, run_oracle, swap_ok

pytestmark = pytest.mark.gpu


def _i16(t):
    import torch

    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def test_l32_32k_every_head_and_three_budgets():
    """32 layers x 8 KV heads x 32768 tokens, W = 64: all 256 heads element by element,
    then the selection at B = 256, 1024 and 4096 (the budget sweep) on the oracle's
    priorities, bit-exact for every head, with the compaction of every head."""
    import torch

    w = make_workload("l32_32k", 233)
    g = HipRun(w)
    log("[full l32_32k] gpu pass")
    sc = g.score(want_saliency=True)
    idx, cu, _ = g.select(sc["scores"])
    torch.cuda.synchronize()
    log("[full l32_32k] oracle, all 256 heads")
    o = run_oracle(w, g.budget, g.params)
    P = sc["scores"].cpu().numpy()
    A = sc["saliency"].cpu().numpy()
    prun = w.protected == 0
    nrow = ref_rows(w, g.budget)[0]
    idx_h = idx.cpu().numpy()[:, :, :nrow]
    for l in range(w.num_layers):
        for h in range(w.num_kv_heads):
            close(P[l, h], o["P"][(0, l, h)], f"P{(l, h)}")
            close(A[l, h], o["A"][(0, l, h)], f"A{(l, h)}")
            swap_ok(idx_h[l, h], o["idx"][(0, l, h)], o["P"][(0, l, h)], prun, g.budget)
    del A, P
    P32 = np.stack([np.stack([o["P"][(0, l, h)] for h in range(w.num_kv_heads)])
                    for l in range(w.num_layers)]).astype(np.float32)
    del o
    Pdev = torch.from_numpy(P32).cuda()
    for budget in (256, 1024, 4096):
        log(f"[full l32_32k] gpu select and compact at B={budget} on oracle priorities")
        idx2, cu2, _ = g.B.select(g.pb, Pdev, g.prot, g.sid, budget)
        rows = int(g.pb.retained_rows(w.protected, budget)[-1])
        assert int(cu2.cpu()[-1]) == rows == O.retained_count(w.seqlens[0], 512, budget)
        k2, v2 = g.B.compact(g.pb, g.k, g.v, idx2, cu2, rows)
        idx2 = idx2.cpu().numpy()
        kh, vh = _i16(k2), _i16(v2)
        for l in range(w.num_layers):
            for h in range(w.num_kv_heads):
                want = O.select_retained(P32[l, h], prun, budget)
                assert np.array_equal(idx2[l, h, :rows], want), (budget, l, h)
                assert np.array_equal(kh[l, h], w.k[l, h][want]), (budget, l, h)
                assert np.array_equal(vh[l, h], w.v[l, h][want]), (budget, l, h)
        del k2, v2, kh, vh
    assert g.pb.status() == 0


def test_l32_16k_sampled():
    """32 layers x 8 KV heads x 16384 tokens, W = 32 (128 window rows, the HBM-bound
    sweep): every head's saliency mass, one head per layer against the oracle element by
    element, and those heads' selection (on the oracle's priorities) and compaction."""
    import torch

    w = make_workload("l32_16k", 233)
    g = HipRun(w)
    log("[full l32_16k] gpu pass")
    sc = g.score(want_saliency=True)
    torch.cuda.synchronize()
    R = w.window * w.group
    A = sc["saliency"].cpu().numpy()
    np.testing.assert_allclose(A.sum(axis=2), R, rtol=1e-4)
    heads = [(l, (3 * l + 1) % w.num_kv_heads) for l in range(w.num_layers)]
    log("[full l32_16k] oracle, one head per layer")
    o = run_oracle(w, g.budget, g.params, heads=heads)
    P = sc["scores"].cpu().numpy()
    prun = w.protected == 0
    P_mix = P.copy()
    for l, h in heads:
        close(P[l, h], o["P"][(0, l, h)], f"P{(l, h)}")
        close(A[l, h], o["A"][(0, l, h)], f"A{(l, h)}")
        P_mix[l, h] = o["P"][(0, l, h)].astype(np.float32)
    idx, cu, _ = g.select(torch.from_numpy(P_mix).cuda())
    k2, v2 = g.compact(idx, cu)
    rows = ref_rows(w, g.budget)[0]
    idx = idx.cpu().numpy()
    kh, vh = _i16(k2), _i16(v2)
    for l, h in heads:
        want = O.select_retained(P_mix[l, h], prun, g.budget)
        assert np.array_equal(idx[l, h, :rows], want), (l, h)
        assert np.array_equal(kh[l, h], w.k[l, h][want]) and np.array_equal(vh[l, h], w.v[l, h][want])
    assert g.pb.status() == 0


def test_ragged16_full_size_with_decode():
    """The ragged batch at full size: 16 sequences of 4k-32k tokens, 28 layers, 4 KV heads,
    G = 7 (224 window rows), B = 2048. Every (sequence, layer, head) saliency mass; one head
    per sequence against the oracle element by element; those heads' selection on the
    oracle's priorities and their compaction bit-exact; and one decode step over the
    compacted cache against textbook attention for every query head of those heads."""
    import torch

    w = make_workload("ragged16", 233)
    g = HipRun(w)
    log(f"[full ragged16] gpu pass, {w.total_tokens} tokens in {w.num_seqs} sequences")
    sc = g.score(want_saliency=True)
    idx_e2e, _, _ = g.select(sc["scores"])
    torch.cuda.synchronize()
    idx_e2e = idx_e2e.cpu().numpy()
    A = sc["saliency"].cpu().numpy()
    R = w.window * w.group
    for s in range(w.num_seqs):
        a, b = int(w.cu_seqlens[s]), int(w.cu_seqlens[s + 1])
        np.testing.assert_allclose(A[:, :, a:b].sum(axis=2), R, rtol=1e-4, err_msg=f"seq {s}")
    picks = [(s, (5 * s + 3) % w.num_layers, s % w.num_kv_heads) for s in range(w.num_seqs)]
    log("[full ragged16] oracle, one head per sequence")
    P = sc["scores"].cpu().numpy()
    P_mix = P.copy()
    prun_all = w.protected == 0
    for s, l, h in picks:
        a, b = int(w.cu_seqlens[s]), int(w.cu_seqlens[s + 1])
        o = run_oracle(w, g.budget, g.params, heads=[(l, h)], seqs=[s])
        close(P[l, h, a:b], o["P"][(s, l, h)], f"P{(s, l, h)}")
        close(A[l, h, a:b], o["A"][(s, l, h)], f"A{(s, l, h)}")
        nk = len(o["idx"][(s, l, h)])
        swap_ok(idx_e2e[l, h, a:a + nk], o["idx"][(s, l, h)], o["P"][(s, l, h)],
                prun_all[a:b], g.budget)
        P_mix[l, h, a:b] = o["P"][(s, l, h)].astype(np.float32)
    del A
    log("[full ragged16] gpu select, compact and decode on oracle priorities")
    idx, cu, _ = g.select(torch.from_numpy(P_mix).cuda())
    k2, v2 = g.compact(idx, cu)
    cu_h = cu.cpu().numpy()
    assert list(cu_h) == list(g.pb.retained_rows(w.protected, g.budget))
    assert list(np.diff(cu_h)) == ref_rows(w, g.budget)
    q_dec = g.B.bf16_from_bits(w.q_dec)
    dec = g.B.decode_attention(g.pb, q_dec, k2, v2, cu, g.out_rows).cpu().numpy()
    idx = idx.cpu().numpy()
    scale = 1.0 / np.sqrt(w.head_dim)
    for s, l, h in picks:
        a, b = int(w.cu_seqlens[s]), int(w.cu_seqlens[s + 1])
        want = O.select_retained(P_mix[l, h, a:b], prun_all[a:b], g.budget)
        r0, r1 = int(cu_h[s]), int(cu_h[s + 1])
        assert np.array_equal(idx[l, h, a:a + (r1 - r0)], want), (s, l, h)
        kh = _i16(k2[l, h, r0:r1])
        vh = _i16(v2[l, h, r0:r1])
        kr, vr = O.compact(w.k[l, h, a:b], w.v[l, h, a:b], want)
        assert np.array_equal(kh, kr) and np.array_equal(vh, vr), (s, l, h)
        for g_ in range(w.group):
            hq = h * w.group + g_
            ref = O.decode_attention(O.decode_bf16(w.q_dec[l, s, hq]), O.decode_bf16(kr),
                                     O.decode_bf16(vr), scale)
            err = np.abs(dec[l, s, hq] - ref).max()
            assert err <= 2e-3 * np.abs(ref).max() + 1e-6, (s, l, hq, err)
    assert g.pb.status() == 0
