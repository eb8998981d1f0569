"""stepkv_score_noalloc (workspace in the library's static device scratch) against
stepkv_score (caller workspace), through the C ABI: two calls in a row, the second on a
smaller problem, each bit-exact with the allocating entry point on the same inputs
(the same kernels run on the same values)."""
import ctypes

import numpy as np
import pytest

from tests.gpu_cases import HipRun, log, reduced

pytestmark = pytest.mark.gpu


def _noalloc(g, scores, sal):
    lib = g.B.load()
    return lib.stepkv_score_noalloc(ctypes.byref(g.pb.c), ctypes.byref(g.params.c()),
                                    g.q.data_ptr(), g.k.data_ptr(), g.sid.data_ptr(),
                                    g.prot.data_ptr(), g.util.data_ptr(), scores.data_ptr(),
                                    sal.data_ptr(), None, g.B._stream(None))


def test_score_noalloc_matches_score_on_two_calls_in_a_row(gpu_lib):
    import torch

    cases = [("l32_32k", dict()),  # the full 32-layer 32k cache: 4.25 MiB of scratch
             ("ragged16", dict(num_layers=2, seqlens=[2500, 700, 130, 1, 0, 4097],
                               protected_len=64))]  # smaller, ragged, G = 7
    for name, kw in cases:
        w = reduced(name, **kw)
        g = HipRun(w, want_v=False)
        need = int(gpu_lib.stepkv_saliency_workspace_bytes(ctypes.byref(g.pb.c)))
        assert 0 < need <= g.B.STATIC_SCRATCH_BYTES
        log(f"[noalloc {name}] L={w.num_layers} tokens={w.total_tokens} scratch={need} bytes")
        shape = (w.num_layers, w.num_kv_heads, w.total_tokens)
        scores = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
        sal = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
        assert _noalloc(g, scores, sal) == 0
        ref = g.score(want_saliency=True)
        torch.cuda.synchronize()
        for got, want, what in ((scores, ref["scores"], "scores"), (sal, ref["saliency"], "A")):
            assert np.array_equal(got.cpu().numpy().view(np.uint32),
                                  want.cpu().numpy().view(np.uint32)), f"{name}: {what}"
        assert g.pb.status() == 0
        log(f"[noalloc {name}] bit-exact with stepkv_score")
