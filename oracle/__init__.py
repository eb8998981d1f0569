"""CPU oracle for StepKV's compression pass (test infrastructure only).

A plain, slow, fp64 numpy restatement of what the compression pass computes,
written from the paper's definitions. Only the test suite, the package smoke
check and the benchmark's CPU-baseline leg may import it; the library under
``paper_2609_22158_amd`` never does, and shares no code with it.

Parity status of each function is listed in ``oracle.stepkv_ref``'s header.
"""
from .stepkv_ref import *  # noqa: F401,F403
from .stepkv_ref import __all__  # noqa: F401
