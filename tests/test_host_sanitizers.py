"""The library's host C++ under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Builds the sanitized variant (paper_2609_22158_amd.build.build_host_sanitized: the host
sources with -fsanitize=address,undefined, linked with the unsanitized HIP objects) and
runs tests/sanitized_host_cases.py in a child process with the sanitizer runtime
preloaded; any sanitizer report ends the child with a nonzero status and fails here.
Skipped on a machine with a visible GPU, where it is not needed and not meant to run."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _gpu_visible():
    try:
        import torch

        return torch.cuda.device_count() > 0
    except Exception:  # pragma: no cover
        return False


@pytest.mark.skipif(_gpu_visible(), reason="a host-only check; runs where no GPU is visible")
def test_host_code_is_clean_under_asan_and_ubsan():
    from paper_2609_22158_amd.build import build_host_sanitized, sanitizer_env

    build_host_sanitized()
    env = sanitizer_env()
    env["PYTHONPATH"] = ROOT + os.pathsep + env.get("PYTHONPATH", "")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "sanitized_host_cases.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-6000:]
    for case in ("check_text_cues", "check_text_engine", "check_step_update",
                 "check_device_call_validation"):
        assert f"{case}: ok" in out, out[-3000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-6000:]
