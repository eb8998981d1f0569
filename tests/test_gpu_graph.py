"""The device part of the compression pass captured in a HIP graph and replayed.

Every entry point launches kernels on the caller's stream and allocates,
copies, clears and synchronizes nothing, so score -> select -> compact can be
recorded once and replayed (the serving-loop use: no launch overhead per
kernel). Each replay, with eager work and a synchronization between replays,
must reproduce the eager results bit for bit.
"""
import ctypes

import numpy as np
import pytest

from tests.gpu_cases import HipRun, log, reduced

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shared", [False, True], ids=["per-head", "shared-index"])
def test_compression_pass_replays_in_a_hip_graph(shared, gpu_lib):
    import torch

    w = reduced("l1_8k", seqlens=[3001, 700, 129])
    g = HipRun(w)
    B, pb = g.B, g.pb
    dev = g.k.device
    L, Hkv, ntot, d = w.num_layers, w.num_kv_heads, w.total_tokens, w.head_dim
    rows = (1 if shared else L * Hkv)
    need = (int(gpu_lib.stepkv_score_shared_workspace_bytes(ctypes.byref(pb.c), 3)) if shared
            else pb.workspace_bytes())
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    scores = torch.empty((ntot,) if shared else (L, Hkv, ntot), dtype=torch.float32, device=dev)
    idx = torch.empty((ntot,) if shared else (L, Hkv, ntot), dtype=torch.int32, device=dev)
    cu_ret = torch.empty(w.num_seqs + 1, dtype=torch.int32, device=dev)
    k_out = torch.empty((L, Hkv, g.out_rows, d), dtype=torch.bfloat16, device=dev)
    v_out = torch.empty_like(k_out)

    def run():
        if shared:
            B.score_shared(pb, g.q, g.k, g.sid, g.prot, g.util, g.params, last_layers=3,
                           workspace=ws, scores=scores)
            B.select_shared(pb, scores, g.prot, g.sid, g.budget, idx=idx, cu_retained=cu_ret)
            B.compact_shared(pb, g.k, g.v, idx, cu_ret, g.out_rows, k_out=k_out, v_out=v_out)
        else:
            B.score(pb, g.q, g.k, g.sid, g.prot, g.util, g.params, workspace=ws, scores=scores)
            B.select(pb, scores, g.prot, g.sid, g.budget, idx=idx, cu_retained=cu_ret)
            B.compact(pb, g.k, g.v, idx, cu_ret, g.out_rows, k_out=k_out, v_out=v_out)

    rows_s = np.diff(pb.retained_rows(w.protected, g.budget))

    def defined(t):  # the entries select writes: the first R_s positions of each sequence
        return torch.cat([t[..., int(w.cu_seqlens[s]):int(w.cu_seqlens[s]) + int(rows_s[s])]
                          for s in range(w.num_seqs)], dim=-1)

    def snapshot():
        torch.cuda.synchronize()
        return [t.clone() for t in (scores, defined(idx), cu_ret, k_out, v_out)]

    log(f"[graph {'shared' if shared else 'per-head'}] rows={rows} eager reference")
    run()
    ref = snapshot()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()  # warm-up on the capturing stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        run()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (scores, idx, k_out, v_out):
            t.zero_()  # eager work between replays (a fill kernel, outside the graph)
        cu_ret.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        got = snapshot()
        for name, a, b in zip(("scores", "idx", "cu_retained", "k_hat", "v_hat"), got, ref):
            if a.dtype == torch.bfloat16:
                a, b = a.view(torch.int16), b.view(torch.int16)
            assert torch.equal(a, b), f"replay {rep}: {name} differs"
        log(f"[graph] replay {rep} matches")
    assert np.array_equal(ref[2].cpu().numpy()[[0, -1]], [0, int(g.out_rows)])
