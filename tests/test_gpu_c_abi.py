"""The C ABI used from plain C, with no Python or torch in the process:
tests/c_abi/compress_demo.c scores, selects and compacts a small two-layer
cache through libstepkv.so and checks the results on the host (saliency mass,
protected tokens, retained counts and order, bit-exact compacted rows)."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

DEMO = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "compress_demo")


def test_plain_c_compression_pass():
    assert os.path.exists(DEMO), "build the library first (it also builds the C demo)"
    print("[c abi] running compress_demo", flush=True)
    r = subprocess.run([DEMO], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stderr
    assert r.stdout.startswith("ok:")
