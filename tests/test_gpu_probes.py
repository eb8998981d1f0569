"""The two measurement probes of the library (not part of the method), checked by what they
must leave behind: the bandwidth probe's copy is the source, and the issue-rate probe with
MFMAs alone does exactly the 4 x iters 32x32x16 products per wave it is timed for.

Issue probe, mix 0: every lane feeds the same eight bf16 values a_j = 0.5 + j/8 as the A
operand and b_j = 1/4 - j/16 as the B operand, so every output of one product is
sum_{k<16} a_{k mod 8} b_{k mod 8} = 2 sum_j a_j b_j; after iters products an accumulator
holds iters times that, exactly (binary fractions well inside fp32). Each thread's sink is
its eight untouched vector values plus the 4 x 16 accumulator entries it holds."""
import numpy as np
import pytest

from tests.gpu_cases import log

pytestmark = pytest.mark.gpu


def test_bandwidth_probe_copies():
    import torch

    from paper_2609_22158_amd import binding as B

    src = torch.randint(0, 255, (3 << 20,), dtype=torch.uint8, device="cuda")
    dst = torch.zeros_like(src)
    log("[probe] bandwidth copy 3 MiB")
    B.bandwidth_probe(src, dst, True)
    assert torch.equal(src, dst)
    B.bandwidth_probe(src, dst, False)  # read only: runs, writes at most bytes / 4096 words
    torch.cuda.synchronize()


@pytest.mark.parametrize("iters", [1, 37, 4000])
def test_issue_probe_does_the_products_it_times(iters):
    import torch

    from paper_2609_22158_amd import binding as B

    blocks = 8
    sink = torch.full((blocks * 256,), float("nan"), dtype=torch.float32, device="cuda")
    log(f"[probe] issue mix 0, {iters} loops")
    B.issue_probe(False, blocks, iters, sink)
    got = sink.cpu().numpy()
    a = np.float32(0.5) + np.float32(0.125) * np.arange(8, dtype=np.float32)
    b = np.float32(0.25) - np.float32(0.0625) * np.arange(8, dtype=np.float32)
    v = np.float32(2.0 * float(np.dot(a.astype(np.float64), b.astype(np.float64))))
    acc = np.float32(0.0)
    for _ in range(iters):
        acc = np.float32(acc + v)
    tid = np.arange(blocks * 256) % 256
    want = np.zeros(blocks * 256, np.float32)
    for i in range(8):
        want += np.float32(1e-3) * np.float32(i + 1) + np.float32(1e-6) * tid.astype(np.float32)
    for _ in range(64):
        want += acc
    np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-6)
    B.issue_probe(True, blocks, iters, sink)  # with the vector mix: runs to the end
    torch.cuda.synchronize()
