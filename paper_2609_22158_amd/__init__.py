"""StepKV compression pass on AMD Instinct MI355X (gfx950).

The pass lives in libstepkv.so (hand-written HIP kernels behind the C ABI of
include/stepkv.h); ``binding`` is its ctypes binding. Importing this package
loads nothing; the first binding call loads the library and raises if it has
not been built.
"""
from . import binding  # noqa: F401
from .binding import (  # noqa: F401
    Params,
    Problem,
    StepKVError,
    StepTracker,
    TextTracker,
    budget_from_ratio,
    compact,
    compact_shared,
    compress,
    decode_attention,
    decode_stats,
    load,
    priority,
    retained_rows,
    saliency,
    saliency_from_lse,
    score,
    score_shared,
    select,
    select_shared,
    step_utilities,
    text_cues,
    window_lse,
)
