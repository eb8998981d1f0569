"""The one-call pass (stepkv_compress), the host retained-row rule and the device status
word, through the C ABI on the GPU.

stepkv_compress must equal stepkv_score -> stepkv_select -> stepkv_compact bit for bit
(it launches the same kernels on one stream); the retained rows computed on the host by
stepkv_retained_rows must equal the cu_retained the selection writes; and every
condition the kernels report (STEPKV_FLAG_*) is planted here from the host into the
inputs, checked to be reported, and checked to leave the defined result unchanged.
"""
import numpy as np
import pytest

import oracle as O
from tests.gpu_cases import HipRun, log, reduced, ref_rows

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": dict(name="tiny"),
    "ragged_g7": dict(name="ragged16", num_layers=2, seqlens=[2500, 700, 130, 1, 0, 4097],
                      protected_len=64),
    "l32_32k_2l": dict(name="l32_32k", num_layers=2, seqlens=[5003], num_steps=20),
}


def _hip(cid, **kw):
    spec = dict(CASES[cid])
    name = spec.pop("name")
    log(f"[compress {cid}] generating")
    return HipRun(reduced(name, **spec), **kw)


def _bits(t):
    import torch

    return t.contiguous().view(torch.int16).cpu().numpy()


@pytest.mark.parametrize("lse_fed", [False, True])
@pytest.mark.parametrize("cid", list(CASES))
def test_compress_equals_the_three_calls(cid, lse_fed):
    import torch

    g = _hip(cid)
    B = g.B
    lse = B.window_lse(g.pb, g.q, g.k, g.params) if lse_fed else None
    log(f"[compress {cid}] one call, lse_fed={lse_fed}")
    one = B.compress(g.pb, g.q, g.k, g.v, g.sid, g.prot, g.util, g.budget, g.out_rows,
                     g.params, lse=lse)
    log(f"[compress {cid}] three calls")
    sc = g.score(lse=lse)
    idx, cu_ret, _ = g.select(sc["scores"])
    k_hat, v_hat = g.compact(idx, cu_ret)
    torch.cuda.synchronize()
    assert np.array_equal(one["scores"].cpu().numpy().view(np.uint32),
                          sc["scores"].cpu().numpy().view(np.uint32))
    assert np.array_equal(one["cu_retained"].cpu().numpy(), cu_ret.cpu().numpy())
    rows = np.diff(cu_ret.cpu().numpy())
    i1, i3 = one["idx"].cpu().numpy(), idx.cpu().numpy()
    for s in range(g.w.num_seqs):  # the defined entries: the first R_s of each sequence
        a = int(g.w.cu_seqlens[s])
        assert np.array_equal(i1[:, :, a:a + rows[s]], i3[:, :, a:a + rows[s]]), s
    assert np.array_equal(_bits(one["k_hat"]), _bits(k_hat))
    assert np.array_equal(_bits(one["v_hat"]), _bits(v_hat))
    # the host rule, the oracle's count and the device selection agree
    host = g.pb.retained_rows(g.w.protected, g.budget)
    assert list(host) == list(cu_ret.cpu().numpy())
    assert list(np.diff(host)) == ref_rows(g.w, g.budget)
    assert g.pb.status() == 0  # clean inputs report nothing


def test_compress_with_per_sequence_budgets_and_workspace_outputs():
    """Per-sequence budgets (one below 1, taken as 1) and scores / idx left in the workspace."""
    import torch

    g = _hip("ragged_g7")
    w = g.w
    budgets = np.array([300, 0, 7, 5, 9, 1200], np.int32)
    cu = g.pb.retained_rows(w.protected, 0, budgets)
    rows = int(cu[-1])
    bud_dev = torch.from_numpy(budgets).cuda()
    lib = g.B.load()
    ws = torch.empty(int(lib.stepkv_compress_workspace_bytes(g.B.ctypes.byref(g.pb.c))),
                     dtype=torch.uint8, device="cuda")
    cu_ret = torch.empty(w.num_seqs + 1, dtype=torch.int32, device="cuda")
    k_out = torch.empty((w.num_layers, w.num_kv_heads, rows, w.head_dim), dtype=torch.bfloat16,
                        device="cuda")
    v_out = torch.empty_like(k_out)
    rc = lib.stepkv_compress(g.B.ctypes.byref(g.pb.c), g.B.ctypes.byref(g.params.c()),
                             g.q.data_ptr(), g.k.data_ptr(), g.v.data_ptr(), None,
                             g.sid.data_ptr(), g.prot.data_ptr(), g.util.data_ptr(), 0,
                             bud_dev.data_ptr(), None, None, cu_ret.data_ptr(), rows,
                             k_out.data_ptr(), v_out.data_ptr(), ws.data_ptr(), ws.numel(),
                             g.B._stream(None))
    assert rc == 0
    sc = g.score()
    idx, cu2, _ = g.select(sc["scores"], budgets=bud_dev)
    k2, v2 = g.B.compact(g.pb, g.k, g.v, idx, cu2, rows)
    torch.cuda.synchronize()
    assert list(cu_ret.cpu().numpy()) == list(cu) == list(cu2.cpu().numpy())
    assert np.array_equal(_bits(k_out), _bits(k2)) and np.array_equal(_bits(v_out), _bits(v2))
    for s in range(w.num_seqs):
        assert cu[s + 1] - cu[s] == O.retained_count(w.seqlens[s], w.protected_len[s],
                                                     max(1, int(budgets[s])))
    assert g.pb.status() == 0


def test_status_reports_step_ids_out_of_range():
    """A prunable token whose step id lies outside [0, n_steps) takes utility 0 and is
    reported; protected tokens (id -1) are not."""
    import torch

    g = _hip("tiny")
    g.pb.status(clear=True)
    g.score()
    assert g.pb.status() == 0
    sid = g.w.step_ids.copy()
    a = int(np.nonzero(g.w.protected == 0)[0][5])
    sid[a] = 10_000
    g.sid = torch.from_numpy(sid).cuda()
    sc = g.score()
    assert g.pb.status(clear=True) == g.B.FLAG_STEP_ID
    assert g.pb.status() == 0  # cleared
    # the result is the defined one: utility 0 for that token
    P = sc["scores"].cpu().numpy()
    sal = g.B.saliency(g.pb, g.q, g.k, g.params)
    ref = g.B.priority(g.pb, sal, g.sid, g.prot, g.util, g.params)["scores"].cpu().numpy()
    assert np.array_equal(P.view(np.uint32), ref.view(np.uint32))
    assert g.pb.status(clear=True) == g.B.FLAG_STEP_ID  # priority alone reports it too


def test_status_reports_non_finite_inputs():
    import torch

    g = _hip("tiny")
    g.pb.status(clear=True)
    k = g.w.k.copy()
    pos = int(np.nonzero(g.w.protected == 0)[0][17])
    k[0, 1, pos, 3] = 0x7FC0  # a NaN in one key of one head
    g.k = g.B.bf16_from_bits(k)
    g.score()
    assert g.pb.status(clear=True) & g.B.FLAG_NONFINITE
    util = g.util_host.copy()
    util[2] = np.inf
    g.k = g.B.bf16_from_bits(g.w.k)
    g.util = torch.from_numpy(util).cuda()
    g.score()
    assert g.pb.status(clear=True) == g.B.FLAG_NONFINITE


def test_status_reports_rows_past_out_rows():
    """A compaction (and a decode) given fewer rows than the selection keeps writes (reads)
    only the rows below out_rows and reports it."""
    import torch

    g = _hip("ragged_g7")
    g.pb.status(clear=True)
    sc = g.score()
    idx, cu_ret, _ = g.select(sc["scores"])
    full_k, full_v = g.compact(idx, cu_ret)
    assert g.pb.status() == 0
    short = g.out_rows - 37
    k_out = torch.zeros((g.w.num_layers, g.w.num_kv_heads, short, g.w.head_dim),
                        dtype=torch.bfloat16, device="cuda")
    v_out = torch.zeros_like(k_out)
    g.B.compact(g.pb, g.k, g.v, idx, cu_ret, short, k_out=k_out, v_out=v_out)
    assert g.pb.status(clear=True) == g.B.FLAG_OUT_ROWS
    assert np.array_equal(_bits(k_out), _bits(full_k[:, :, :short]))
    assert np.array_equal(_bits(v_out), _bits(full_v[:, :, :short]))
    # out_rows = 0: nothing is written, the condition is still reported
    g.B.compact(g.pb, g.k, g.v, idx, cu_ret, 0)
    assert g.pb.status(clear=True) == g.B.FLAG_OUT_ROWS
    q_dec = g.B.bf16_from_bits(g.w.q_win[:, :, 0])
    g.B.decode_attention(g.pb, q_dec, k_out, v_out, cu_ret, short)
    assert g.pb.status(clear=True) == g.B.FLAG_OUT_ROWS
    g.B.decode_attention(g.pb, q_dec, full_k, full_v, cu_ret, g.out_rows)
    assert g.pb.status() == 0


def test_status_in_shared_index_mode():
    import torch

    g = _hip("ragged_g7")
    g.pb.status(clear=True)
    g.B.score_shared(g.pb, g.q, g.k, g.sid, g.prot, g.util, g.params, last_layers=2)
    assert g.pb.status() == 0
    sid = g.w.step_ids.copy()
    pos = int(np.nonzero(g.w.protected == 0)[0][-3])
    sid[pos] = -5
    sid_dev = torch.from_numpy(sid).cuda()
    g.B.score_shared(g.pb, g.q, g.k, sid_dev, g.prot, g.util, g.params, last_layers=2)
    assert g.pb.status(clear=True) == g.B.FLAG_STEP_ID
    g.B.score_shared(g.pb, g.q, g.k, sid_dev, g.prot, g.util, g.params, last_layers=2,
                     want_stats=True)  # the one-workgroup priority path
    assert g.pb.status(clear=True) == g.B.FLAG_STEP_ID
