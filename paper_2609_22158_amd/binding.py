"""ctypes binding of libstepkv.so (the C ABI declared in include/stepkv.h).

Argument marshalling only: every step of the compression pass runs in the
library's HIP kernels. PyTorch supplies device memory and the current stream.
There is no CPU fallback; a missing library raises at load time.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libstepkv.so")

OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EHIP, ESCRATCH = 0, -1, -2, -3, -4, -5
STATIC_SCRATCH_BYTES = 128 << 20  # STEPKV_STATIC_SCRATCH_BYTES
FLAG_STEP_ID, FLAG_NONFINITE, FLAG_OUT_ROWS, FLAG_SYNC = 1, 2, 4, 8  # STEPKV_FLAG_*
CUE_CAP = 64  # STEPKV_CUE_CAP
MAX_WINDOW_ROWS = 2048
MAX_POOL_KERNEL = 63
MAX_STEPS_STATS = 4096

_i32p = ctypes.POINTER(ctypes.c_int32)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_vp = ctypes.c_void_p


class ProblemC(ctypes.Structure):
    _fields_ = [
        ("num_layers", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("num_seqs", ctypes.c_int32),
        ("cu_seqlens_host", _i32p),
        ("cu_seqlens", _vp),
        ("cu_steps_host", _i32p),
        ("cu_steps", _vp),
        ("status", _vp),
    ]


class ParamsC(ctypes.Structure):
    _fields_ = [
        ("alpha", ctypes.c_float),
        ("beta", ctypes.c_float),
        ("pool_kernel", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("lambda_red", ctypes.c_float),
        ("w_r", ctypes.c_float),
        ("w_c", ctypes.c_float),
        ("r_min", ctypes.c_float),
        ("r_max", ctypes.c_float),
        ("s_max", ctypes.c_float),
        ("eta", ctypes.c_float),
        ("causal_tail", ctypes.c_int32),
        ("saliency_schedule", ctypes.c_int32),
    ]


class StepStatC(ctypes.Structure):
    _fields_ = [
        ("count", ctypes.c_uint32),
        ("max_saliency", ctypes.c_float),
        ("sum_saliency_q32", ctypes.c_uint64),
    ]


class StepStateC(ctypes.Structure):
    _fields_ = [
        ("capacity", ctypes.c_int32),
        ("num_steps", ctypes.c_int32),
        ("r", _f64p),
        ("c", _f64p),
    ]


_SIGNATURES = {
    "stepkv_params_default": (None, [ctypes.POINTER(ParamsC)]),
    "stepkv_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "stepkv_budget_from_ratio": (ctypes.c_int64, [ctypes.c_double, ctypes.c_int64]),
    "stepkv_step_update": (ctypes.c_int, [ctypes.POINTER(StepStateC), ctypes.c_float,
                                          ctypes.c_float, ctypes.c_float, _f32p,
                                          ctypes.POINTER(ParamsC), _f32p]),
    "stepkv_text_state_bytes": (ctypes.c_size_t, [ctypes.c_int32]),
    "stepkv_text_state_init": (ctypes.c_int, [_vp, ctypes.c_size_t, ctypes.c_int32]),
    "stepkv_text_step": (ctypes.c_int, [_vp, ctypes.c_char_p, ctypes.c_int64, ctypes.c_char_p,
                                        ctypes.c_int64, ctypes.c_char_p, ctypes.c_int64, _f32p,
                                        _f32p, _f32p, _f32p]),
    "stepkv_text_cues": (ctypes.c_int, [ctypes.c_char_p, ctypes.c_int64,
                                        ctypes.POINTER(ctypes.c_uint64),
                                        ctypes.POINTER(ctypes.c_int32)]),
    "stepkv_retained_rows": (ctypes.c_int, [ctypes.POINTER(ProblemC), _vp, ctypes.c_int32, _vp,
                                            _vp]),
    "stepkv_status_read": (ctypes.c_int, [ctypes.POINTER(ProblemC),
                                          ctypes.POINTER(ctypes.c_uint32), ctypes.c_int32, _vp]),
    "stepkv_compress_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(ProblemC)]),
    "stepkv_score_noalloc": (ctypes.c_int, [ctypes.POINTER(ProblemC), ctypes.POINTER(ParamsC),
                                            _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "stepkv_compress": (ctypes.c_int, [ctypes.POINTER(ProblemC), ctypes.POINTER(ParamsC), _vp, _vp,
                                       _vp, _vp, _vp, _vp, _vp, ctypes.c_int32, _vp, _vp, _vp,
                                       _vp, ctypes.c_int32, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "stepkv_bandwidth_probe": (ctypes.c_int, [_vp, _vp, ctypes.c_size_t, ctypes.c_int32, _vp]),
    "stepkv_issue_probe": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp,
                                          _vp]),
    "stepkv_score_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(ProblemC)]),
    "stepkv_saliency_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(ProblemC)]),
    "stepkv_saliency": (ctypes.c_int, [ctypes.POINTER(ProblemC), ctypes.POINTER(ParamsC), _vp,
                                       _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "stepkv_priority": (ctypes.c_int, [ctypes.POINTER(ProblemC), ctypes.POINTER(ParamsC), _vp,
                                       _vp, _vp, _vp, _vp, _vp, _vp]),
    "stepkv_score": (ctypes.c_int, [ctypes.POINTER(ProblemC), ctypes.POINTER(ParamsC), _vp, _vp,
                                    _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "stepkv_window_lse": (ctypes.c_int, [ctypes.POINTER(ProblemC), ctypes.POINTER(ParamsC), _vp,
                                         _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "stepkv_saliency_from_lse": (ctypes.c_int, [ctypes.POINTER(ProblemC), ctypes.POINTER(ParamsC),
                                                _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "stepkv_score_from_lse": (ctypes.c_int, [ctypes.POINTER(ProblemC), ctypes.POINTER(ParamsC),
                                             _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                             ctypes.c_size_t, _vp]),
    "stepkv_score_shared_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(ProblemC),
                                                            ctypes.c_int32]),
    "stepkv_score_shared": (ctypes.c_int, [ctypes.POINTER(ProblemC), ctypes.POINTER(ParamsC), _vp,
                                           _vp, _vp, ctypes.c_int32, _vp, _vp, _vp, _vp, _vp,
                                           _vp, _vp, ctypes.c_size_t, _vp]),
    "stepkv_select_shared": (ctypes.c_int, [ctypes.POINTER(ProblemC), _vp, _vp, _vp,
                                            ctypes.c_int32, _vp, _vp, _vp, _vp, _vp]),
    "stepkv_compact_shared": (ctypes.c_int, [ctypes.POINTER(ProblemC), _vp, _vp, _vp, _vp,
                                             ctypes.c_int32, _vp, _vp, _vp]),
    "stepkv_select": (ctypes.c_int, [ctypes.POINTER(ProblemC), _vp, _vp, _vp, ctypes.c_int32,
                                     _vp, _vp, _vp, _vp, _vp]),
    "stepkv_compact": (ctypes.c_int, [ctypes.POINTER(ProblemC), _vp, _vp, _vp, _vp,
                                      ctypes.c_int32, _vp, _vp, _vp]),
    "stepkv_decode_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(ProblemC), ctypes.c_int32]),
    "stepkv_decode_attention": (ctypes.c_int, [ctypes.POINTER(ProblemC), _vp, _vp, _vp, _vp,
                                               ctypes.c_int32, ctypes.c_float, _vp, _vp,
                                               ctypes.c_size_t, _vp]),
}

_lib: Optional[ctypes.CDLL] = None


class StepKVError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn} failed: {code} ({strerror(code)})")
        self.code = code


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libstepkv.so and declare its signatures; raises if it is missing.

    The path defaults to the in-tree build; STEPKV_LIB names another build.
    """
    global _lib
    if _lib is not None:
        return _lib
    path = path or os.environ.get("STEPKV_LIB") or LIB_PATH
    if not os.path.exists(path):
        raise ImportError(
            f"{path} not found: build it with `python -m paper_2609_22158_amd.build` "
            "(hipcc, gfx950); there is no fallback implementation")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def strerror(code: int) -> str:
    return load().stepkv_strerror(code).decode()


def _check(fn: str, rc: int) -> None:
    if rc != OK:
        raise StepKVError(fn, rc)


# ---------------------------------------------------------------- parameters
@dataclass
class Params:
    """Method parameters; defaults are the paper's (filled by the library)."""

    alpha: float = 0.2
    beta: float = 0.8
    pool_kernel: int = 7
    scale: float = 0.0  # <= 0: 1/sqrt(d)
    lambda_red: float = 0.3
    w_r: float = 0.85
    w_c: float = 0.15
    r_min: float = -1.0
    r_max: float = 2.0
    s_max: float = 8.0
    eta: float = 1.5
    causal_tail: int = 0  # nonzero: window slot w sees keys 0 .. N - W + w only
    saliency_schedule: int = 0  # 0 per problem, 1 one launch per sweep, 2 both in one launch

    def c(self) -> ParamsC:
        return ParamsC(*[getattr(self, f) for f, _ in ParamsC._fields_])

    @staticmethod
    def token_only(pool_kernel: int = 7, **kw) -> "Params":
        """A token-only selector on the same pass: the retention priority is the pooled
        window saliency alone (beta = 0), as in the paper's 'w/o step score' ablation
        (Table 3). With the default window this is a SnapKV-style selector."""
        return Params(alpha=1.0, beta=0.0, pool_kernel=pool_kernel, **kw)

    @staticmethod
    def last_query_only(**kw) -> "Params":
        """The TOVA-style selector: with a window of one query (W = 1 in the problem),
        no pooling and beta = 0, tokens rank by the newest query's attention."""
        return Params(alpha=1.0, beta=0.0, pool_kernel=1, **kw)

    @staticmethod
    def library_default() -> "Params":
        p = ParamsC()
        load().stepkv_params_default(ctypes.byref(p))
        return Params(**{f: getattr(p, f) for f, _ in ParamsC._fields_})


def budget_from_ratio(rho: float, n_prunable: int) -> int:
    return int(load().stepkv_budget_from_ratio(float(rho), int(n_prunable)))


def step_utilities(valid: Sequence[float], gain: Sequence[float], red: Sequence[float],
                   obs_sim: np.ndarray, params: Optional[Params] = None) -> np.ndarray:
    """Run the host step-utility update over boundaries 1..n; returns S (float32 [n])."""
    lib = load()
    p = (params or Params()).c()
    n = len(valid)
    r = np.zeros(max(n, 1), np.float64)
    c = np.zeros(max(n, 1), np.float64)
    st = StepStateC(max(n, 1), 0, r.ctypes.data_as(_f64p), c.ctypes.data_as(_f64p))
    S = np.zeros(max(n, 1), np.float32)
    sim = np.ascontiguousarray(obs_sim, dtype=np.float32)
    for t in range(n):
        row = np.ascontiguousarray(sim[t, :t]) if t > 0 else None
        rc = lib.stepkv_step_update(ctypes.byref(st), float(valid[t]), float(gain[t]),
                                    float(red[t]),
                                    row.ctypes.data_as(_f32p) if row is not None else None,
                                    ctypes.byref(p), S.ctypes.data_as(_f32p))
        _check("stepkv_step_update", rc)
    return S[:n].copy()


class StepTracker:
    """Step-utility state of one trajectory across pruning boundaries (Algorithm 1
    phases 1-2, one stepkv_step_update per boundary). `update` adds step t and
    returns (or writes into `out`) the utilities S_0..S_t as float32."""

    def __init__(self, capacity: int, params: Optional[Params] = None):
        self.capacity = max(int(capacity), 1)
        self.r = np.zeros(self.capacity, np.float64)
        self.c = np.zeros(self.capacity, np.float64)
        self.S = np.zeros(self.capacity, np.float32)
        self._p = (params or Params()).c()
        self._st = StepStateC(self.capacity, 0, self.r.ctypes.data_as(_f64p),
                              self.c.ctypes.data_as(_f64p))

    @property
    def num_steps(self) -> int:
        return int(self._st.num_steps)

    def update(self, valid: float, gain: float, red: float, sim_prev=None, out=None) -> np.ndarray:
        """Boundary after step t = num_steps: sim_prev[k] = sim(Obs_t, Obs_k) for k < t."""
        t = self.num_steps
        row = None
        if t > 0:
            row = np.ascontiguousarray(sim_prev, dtype=np.float32)
            if row.shape != (t,):
                raise ValueError(f"sim_prev: shape {row.shape}, expected ({t},)")
        dst = self.S if out is None else out
        if out is not None and (out.dtype != np.float32 or not out.flags.c_contiguous
                                or out.shape[0] < t + 1):
            raise ValueError("out: a contiguous float32 array of at least t + 1 entries")
        rc = load().stepkv_step_update(ctypes.byref(self._st), float(valid), float(gain),
                                       float(red), row.ctypes.data_as(_f32p) if row is not None
                                       else None, ctypes.byref(self._p),
                                       dst.ctypes.data_as(_f32p))
        _check("stepkv_step_update", rc)
        return dst[:t + 1]

    def snapshot(self):
        return self.r.copy(), self.c.copy(), self.num_steps

    def restore(self, snap) -> None:
        r, c, n = snap
        self.r[:] = r
        self.c[:] = c
        self._st.num_steps = n


def _text(x) -> bytes:
    return x if isinstance(x, bytes) else str(x).encode("utf-8")


def text_cues(text) -> np.ndarray:
    """stepkv_text_cues: the cues of one text as uint64 FNV-1a hashes, in order."""
    data = _text(text)
    out = (ctypes.c_uint64 * CUE_CAP)()
    n = ctypes.c_int32(0)
    _check("stepkv_text_cues", load().stepkv_text_cues(data, len(data), out, ctypes.byref(n)))
    return np.array(out[:n.value], dtype=np.uint64)


class TextTracker:
    """Step signals of one trajectory from its text (stepkv_text_step), optionally fed
    straight into the utilities (StepTracker): `signals` adds a step and returns
    (valid, gain, red, obs_sim_prev); `update` also advances the utilities and returns S."""

    def __init__(self, capacity: int, params: Optional[Params] = None):
        lib = load()
        self.capacity = max(int(capacity), 1)
        nbytes = int(lib.stepkv_text_state_bytes(self.capacity))
        self._nbytes = nbytes
        self._state = np.zeros((nbytes + 7) // 8, np.uint64)  # 8-byte aligned host memory
        _check("stepkv_text_state_init",
               lib.stepkv_text_state_init(self._state.ctypes.data, nbytes, self.capacity))
        self.steps = StepTracker(self.capacity, params)
        self._sim = np.zeros(self.capacity, np.float32)

    @property
    def num_steps(self) -> int:
        return int(self._state[:2].view(np.int32)[2])  # the state header's step count

    def signals(self, thought, action, observation):
        t = self.num_steps
        th, ac, ob = _text(thought), _text(action), _text(observation)
        v, g, r = ctypes.c_float(), ctypes.c_float(), ctypes.c_float()
        rc = load().stepkv_text_step(self._state.ctypes.data, th, len(th), ac, len(ac), ob, len(ob),
                                     ctypes.byref(v), ctypes.byref(g), ctypes.byref(r),
                                     self._sim.ctypes.data_as(_f32p))
        _check("stepkv_text_step", rc)
        return v.value, g.value, r.value, self._sim[:t].copy()

    def update(self, thought, action, observation, out=None) -> np.ndarray:
        v, g, r, sim = self.signals(thought, action, observation)
        return self.steps.update(v, g, r, sim, out=out)

    def snapshot(self):
        return self._state.copy(), self.steps.snapshot()

    def restore(self, snap) -> None:
        self._state[:] = snap[0]
        self.steps.restore(snap[1])


# ---------------------------------------------------------------- problem
class Problem:
    """Shape of one compression problem with host and device offset arrays."""

    def __init__(self, num_layers: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
                 window: int, cu_seqlens, cu_steps, device="cuda", status: bool = True):
        import torch

        self.cu_seqlens = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
        self.cu_steps = np.ascontiguousarray(cu_steps, dtype=np.int32)
        self.num_seqs = int(self.cu_seqlens.shape[0] - 1)
        self.cu_seqlens_dev = torch.from_numpy(self.cu_seqlens).to(device)
        self.cu_steps_dev = torch.from_numpy(self.cu_steps).to(device)
        self.num_layers, self.num_q_heads, self.num_kv_heads = num_layers, num_q_heads, num_kv_heads
        self.head_dim, self.window = head_dim, window
        self.device = device
        # the device status word the kernels report conditions into (STEPKV_FLAG_*)
        self.status_dev = torch.zeros(1, dtype=torch.int32, device=device) if status else None
        self.c = ProblemC(num_layers, num_q_heads, num_kv_heads, head_dim, window, self.num_seqs,
                          self.cu_seqlens.ctypes.data_as(_i32p), self.cu_seqlens_dev.data_ptr(),
                          self.cu_steps.ctypes.data_as(_i32p), self.cu_steps_dev.data_ptr(),
                          self.status_dev.data_ptr() if status else None)

    def status(self, clear: bool = False, stream=None) -> int:
        """stepkv_status_read: the STEPKV_FLAG_* bits reported so far (waits for the stream)."""
        flags = ctypes.c_uint32(0)
        _check("stepkv_status_read", load().stepkv_status_read(
            ctypes.byref(self.c), ctypes.byref(flags), int(bool(clear)), _stream(stream)))
        return int(flags.value)

    def retained_rows(self, protected, budget: int, budgets=None) -> np.ndarray:
        """stepkv_retained_rows: cu_retained [S+1] (host int32) for a host protected mask;
        its last entry is the out_rows that compaction needs."""
        return retained_rows(self, protected, budget, budgets)

    @classmethod
    def from_workload(cls, w, device="cuda", status: bool = True) -> "Problem":
        return cls(w.num_layers, w.num_q_heads, w.num_kv_heads, w.head_dim, w.window,
                   w.cu_seqlens, w.cu_steps, device, status)

    @property
    def ntot(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def total_steps(self) -> int:
        return int(self.cu_steps[-1])

    @property
    def lh(self) -> int:
        return self.num_layers * self.num_kv_heads

    def workspace_bytes(self) -> int:
        return int(load().stepkv_score_workspace_bytes(ctypes.byref(self.c)))

    def saliency_workspace_bytes(self) -> int:
        return int(load().stepkv_saliency_workspace_bytes(ctypes.byref(self.c)))


def _stream(stream) -> int:
    import torch

    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _need(t, dtype, shape, name):
    import torch

    if t.dtype != dtype:
        raise TypeError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous() or t.device.type != "cuda":
        raise ValueError(f"{name}: must be a contiguous CUDA tensor")
    return t.data_ptr()


def score(pb: Problem, q_win, k, step_ids, protected, step_utility, params: Optional[Params] = None,
          *, lse=None, want_saliency: bool = False, want_stats: bool = False, workspace=None,
          scores=None, stream=None):
    """stepkv_score: priorities P [L*Hkv][Ntot] (and optionally A and step stats).

    With `lse` (fp32 [L][S][W][Hq], the window rows' natural-log log-sum-exps)
    this is stepkv_score_from_lse: one sweep over K instead of two.
    """
    import torch

    lib = load()
    L, Hkv, d, W, S = pb.num_layers, pb.num_kv_heads, pb.head_dim, pb.window, pb.num_seqs
    dev = pb.device
    qp = _need(q_win, torch.bfloat16, (L, S, W, pb.num_q_heads, d), "q_win")
    kp = _need(k, torch.bfloat16, (L, Hkv, pb.ntot, d), "k")
    lp = _need(lse, torch.float32, (L, S, W, pb.num_q_heads), "lse") if lse is not None else None
    sp = _need(step_ids, torch.int32, (pb.ntot,), "step_ids")
    pp = _need(protected, torch.uint8, (pb.ntot,), "protected")
    up = _need(step_utility, torch.float32, (pb.total_steps,), "step_utility")
    if scores is None:
        scores = torch.empty((L, Hkv, pb.ntot), dtype=torch.float32, device=dev)
    out = {"scores": scores}
    sal = torch.empty((L, Hkv, pb.ntot), dtype=torch.float32, device=dev) if want_saliency else None
    stats = (torch.empty((L, Hkv, pb.total_steps, 2), dtype=torch.int64, device=dev)
             if want_stats else None)
    need = pb.workspace_bytes()
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    tail = (scores.data_ptr(), sal.data_ptr() if sal is not None else None,
            stats.data_ptr() if stats is not None else None, workspace.data_ptr(),
            workspace.numel(), _stream(stream))
    prm = ctypes.byref((params or Params()).c())
    if lp is None:
        _check("stepkv_score", lib.stepkv_score(ctypes.byref(pb.c), prm, qp, kp, sp, pp, up, *tail))
    else:
        _check("stepkv_score_from_lse",
               lib.stepkv_score_from_lse(ctypes.byref(pb.c), prm, qp, kp, lp, sp, pp, up, *tail))
    if sal is not None:
        out["saliency"] = sal
    if stats is not None:
        out["stats_raw"] = stats
    return out


def saliency(pb: Problem, q_win, k, params: Optional[Params] = None, *, workspace=None, out=None,
             stream=None):
    """stepkv_saliency: raw window saliency A [L][Hkv][Ntot] (fp32)."""
    import torch

    lib = load()
    L, Hkv, d, W, S = pb.num_layers, pb.num_kv_heads, pb.head_dim, pb.window, pb.num_seqs
    qp = _need(q_win, torch.bfloat16, (L, S, W, pb.num_q_heads, d), "q_win")
    kp = _need(k, torch.bfloat16, (L, Hkv, pb.ntot, d), "k")
    if out is None:
        out = torch.empty((L, Hkv, pb.ntot), dtype=torch.float32, device=pb.device)
    _need(out, torch.float32, (L, Hkv, pb.ntot), "saliency")
    if workspace is None:
        workspace = torch.empty(max(pb.saliency_workspace_bytes(), 1), dtype=torch.uint8,
                                device=pb.device)
    rc = lib.stepkv_saliency(ctypes.byref(pb.c), ctypes.byref((params or Params()).c()), qp, kp,
                             out.data_ptr(), workspace.data_ptr(), workspace.numel(),
                             _stream(stream))
    _check("stepkv_saliency", rc)
    return out


def window_lse(pb: Problem, q_win, k, params: Optional[Params] = None, *, workspace=None,
               out=None, stream=None):
    """stepkv_window_lse: natural-log row log-sum-exp of the window attention, [L][S][W][Hq]."""
    import torch

    lib = load()
    L, Hkv, d, W, S = pb.num_layers, pb.num_kv_heads, pb.head_dim, pb.window, pb.num_seqs
    qp = _need(q_win, torch.bfloat16, (L, S, W, pb.num_q_heads, d), "q_win")
    kp = _need(k, torch.bfloat16, (L, Hkv, pb.ntot, d), "k")
    if out is None:
        out = torch.empty((L, S, W, pb.num_q_heads), dtype=torch.float32, device=pb.device)
    op = _need(out, torch.float32, (L, S, W, pb.num_q_heads), "lse")
    if workspace is None:
        workspace = torch.empty(max(pb.saliency_workspace_bytes(), 1), dtype=torch.uint8,
                                device=pb.device)
    rc = lib.stepkv_window_lse(ctypes.byref(pb.c), ctypes.byref((params or Params()).c()), qp, kp,
                               op, workspace.data_ptr(), workspace.numel(), _stream(stream))
    _check("stepkv_window_lse", rc)
    return out


def saliency_from_lse(pb: Problem, q_win, k, lse, params: Optional[Params] = None, *,
                      workspace=None, out=None, stream=None):
    """stepkv_saliency_from_lse: A [L][Hkv][Ntot] in one sweep, given the rows' LSE."""
    import torch

    lib = load()
    L, Hkv, d, W, S = pb.num_layers, pb.num_kv_heads, pb.head_dim, pb.window, pb.num_seqs
    qp = _need(q_win, torch.bfloat16, (L, S, W, pb.num_q_heads, d), "q_win")
    kp = _need(k, torch.bfloat16, (L, Hkv, pb.ntot, d), "k")
    lp = _need(lse, torch.float32, (L, S, W, pb.num_q_heads), "lse")
    if out is None:
        out = torch.empty((L, Hkv, pb.ntot), dtype=torch.float32, device=pb.device)
    _need(out, torch.float32, (L, Hkv, pb.ntot), "saliency")
    if workspace is None:
        workspace = torch.empty(max(pb.saliency_workspace_bytes(), 1), dtype=torch.uint8,
                                device=pb.device)
    rc = lib.stepkv_saliency_from_lse(ctypes.byref(pb.c), ctypes.byref((params or Params()).c()),
                                      qp, kp, lp, out.data_ptr(), workspace.data_ptr(),
                                      workspace.numel(), _stream(stream))
    _check("stepkv_saliency_from_lse", rc)
    return out


def priority(pb: Problem, sal, step_ids, protected, step_utility,
             params: Optional[Params] = None, *, want_stats: bool = False, scores=None,
             stream=None):
    """stepkv_priority: P [L][Hkv][Ntot] from a saliency (and optionally step stats)."""
    import torch

    lib = load()
    L, Hkv = pb.num_layers, pb.num_kv_heads
    ap = _need(sal, torch.float32, (L, Hkv, pb.ntot), "saliency")
    sp = _need(step_ids, torch.int32, (pb.ntot,), "step_ids")
    pp = _need(protected, torch.uint8, (pb.ntot,), "protected")
    up = _need(step_utility, torch.float32, (pb.total_steps,), "step_utility")
    if scores is None:
        scores = torch.empty((L, Hkv, pb.ntot), dtype=torch.float32, device=pb.device)
    _need(scores, torch.float32, (L, Hkv, pb.ntot), "scores")
    stats = (torch.empty((L, Hkv, pb.total_steps, 2), dtype=torch.int64, device=pb.device)
             if want_stats else None)
    rc = lib.stepkv_priority(ctypes.byref(pb.c), ctypes.byref((params or Params()).c()), ap, sp,
                             pp, up, scores.data_ptr(),
                             stats.data_ptr() if stats is not None else None, _stream(stream))
    _check("stepkv_priority", rc)
    out = {"scores": scores}
    if stats is not None:
        out["stats_raw"] = stats
    return out


def score_shared(pb: Problem, q_win, k, step_ids, protected, step_utility,
                 params: Optional[Params] = None, *, last_layers: int = 3, lse=None,
                 want_saliency: bool = False, want_stats: bool = False, workspace=None,
                 scores=None, stream=None):
    """stepkv_score_shared: one priority row per sequence, P [Ntot], from the saliency of
    the last `last_layers` layers summed over their KV heads (optionally from row LSEs)."""
    import torch

    lib = load()
    L, Hkv, d, W, S = pb.num_layers, pb.num_kv_heads, pb.head_dim, pb.window, pb.num_seqs
    dev = pb.device
    qp = _need(q_win, torch.bfloat16, (L, S, W, pb.num_q_heads, d), "q_win")
    kp = _need(k, torch.bfloat16, (L, Hkv, pb.ntot, d), "k")
    lp = _need(lse, torch.float32, (L, S, W, pb.num_q_heads), "lse") if lse is not None else None
    sp = _need(step_ids, torch.int32, (pb.ntot,), "step_ids")
    pp = _need(protected, torch.uint8, (pb.ntot,), "protected")
    up = _need(step_utility, torch.float32, (pb.total_steps,), "step_utility")
    if scores is None:
        scores = torch.empty(pb.ntot, dtype=torch.float32, device=dev)
    _need(scores, torch.float32, (pb.ntot,), "scores")
    sal = torch.empty(pb.ntot, dtype=torch.float32, device=dev) if want_saliency else None
    stats = (torch.empty((pb.total_steps, 2), dtype=torch.int64, device=dev)
             if want_stats else None)
    if workspace is None:
        need = int(lib.stepkv_score_shared_workspace_bytes(ctypes.byref(pb.c), last_layers))
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    rc = lib.stepkv_score_shared(ctypes.byref(pb.c), ctypes.byref((params or Params()).c()), qp,
                                 kp, lp, last_layers, sp, pp, up, scores.data_ptr(),
                                 sal.data_ptr() if sal is not None else None,
                                 stats.data_ptr() if stats is not None else None,
                                 workspace.data_ptr(), workspace.numel(), _stream(stream))
    _check("stepkv_score_shared", rc)
    out = {"scores": scores}
    if sal is not None:
        out["saliency"] = sal
    if stats is not None:
        out["stats_raw"] = stats
    return out


def select_shared(pb: Problem, scores, protected, step_ids, budget: int, *, budgets=None,
                  want_kept: bool = False, idx=None, cu_retained=None, stream=None):
    """stepkv_select_shared: one retained set per sequence, idx [Ntot]."""
    import torch

    lib = load()
    dev = pb.device
    sp_ = _need(scores, torch.float32, (pb.ntot,), "scores")
    pp = _need(protected, torch.uint8, (pb.ntot,), "protected")
    ip = _need(step_ids, torch.int32, (pb.ntot,), "step_ids")
    bp = _need(budgets, torch.int32, (pb.num_seqs,), "budgets") if budgets is not None else None
    if idx is None:
        idx = torch.empty(pb.ntot, dtype=torch.int32, device=dev)
    if cu_retained is None:
        cu_retained = torch.empty(pb.num_seqs + 1, dtype=torch.int32, device=dev)
    kept = torch.empty(pb.total_steps, dtype=torch.int32, device=dev) if want_kept else None
    rc = lib.stepkv_select_shared(ctypes.byref(pb.c), sp_, pp, ip, int(budget), bp,
                                  idx.data_ptr(), cu_retained.data_ptr(),
                                  kept.data_ptr() if kept is not None else None, _stream(stream))
    _check("stepkv_select_shared", rc)
    out = {"idx": idx, "cu_retained": cu_retained}
    if kept is not None:
        out["kept"] = kept
    return out


def compact_shared(pb: Problem, k, v, idx, cu_retained, out_rows: int, *, k_out=None, v_out=None,
                   stream=None):
    """stepkv_compact_shared: every (layer, KV head) gathers the same positions idx [Ntot]."""
    import torch

    lib = load()
    L, Hkv, d = pb.num_layers, pb.num_kv_heads, pb.head_dim
    kp = _need(k, torch.bfloat16, (L, Hkv, pb.ntot, d), "k")
    vp = _need(v, torch.bfloat16, (L, Hkv, pb.ntot, d), "v")
    ip = _need(idx, torch.int32, (pb.ntot,), "idx")
    cp = _need(cu_retained, torch.int32, (pb.num_seqs + 1,), "cu_retained")
    if k_out is None:
        k_out = torch.empty((L, Hkv, out_rows, d), dtype=torch.bfloat16, device=pb.device)
    if v_out is None:
        v_out = torch.empty_like(k_out)
    _need(k_out, torch.bfloat16, (L, Hkv, out_rows, d), "k_out")
    _need(v_out, torch.bfloat16, (L, Hkv, out_rows, d), "v_out")
    rc = lib.stepkv_compact_shared(ctypes.byref(pb.c), kp, vp, ip, cp, int(out_rows),
                                   k_out.data_ptr(), v_out.data_ptr(), _stream(stream))
    _check("stepkv_compact_shared", rc)
    return k_out, v_out


def decode_stats(stats_raw) -> dict:
    """Split the packed stepkv_step_stat records into count / max / sum arrays (host)."""
    raw = stats_raw.cpu().numpy().reshape(-1, 2)
    lo = raw[:, 0].view(np.uint64)
    count = (lo & np.uint64(0xFFFFFFFF)).astype(np.int64)
    mx = (lo >> np.uint64(32)).astype(np.uint32).view(np.float32)
    sm = raw[:, 1].view(np.uint64).astype(np.float64) / 2.0**32
    shape = stats_raw.shape[:-1]
    return {"count": count.reshape(shape), "max": mx.reshape(shape), "sum": sm.reshape(shape)}


def select(pb: Problem, scores, protected, step_ids, budget: int, *, budgets=None,
           want_kept: bool = False, idx=None, cu_retained=None, stream=None):
    """stepkv_select: idx [L][Hkv][Ntot] (sequence s at cu_seqlens[s]) and cu_retained [S+1]."""
    import torch

    lib = load()
    L, Hkv, dev = pb.num_layers, pb.num_kv_heads, pb.device
    scp = _need(scores, torch.float32, (L, Hkv, pb.ntot), "scores")
    pp = _need(protected, torch.uint8, (pb.ntot,), "protected")
    sp = _need(step_ids, torch.int32, (pb.ntot,), "step_ids")
    bp = _need(budgets, torch.int32, (pb.num_seqs,), "budgets") if budgets is not None else None
    if idx is None:
        idx = torch.empty((L, Hkv, pb.ntot), dtype=torch.int32, device=dev)
    _need(idx, torch.int32, (L, Hkv, pb.ntot), "idx")
    cu_ret = cu_retained
    if cu_ret is None:
        cu_ret = torch.empty(pb.num_seqs + 1, dtype=torch.int32, device=dev)
    _need(cu_ret, torch.int32, (pb.num_seqs + 1,), "cu_retained")
    kept = torch.empty((L, Hkv, pb.total_steps), dtype=torch.int32, device=dev) if want_kept else None
    rc = lib.stepkv_select(ctypes.byref(pb.c), scp, pp, sp, int(budget), bp, idx.data_ptr(),
                           cu_ret.data_ptr(), kept.data_ptr() if kept is not None else None,
                           _stream(stream))
    _check("stepkv_select", rc)
    return idx, cu_ret, kept


def compact(pb: Problem, k, v, idx, cu_retained, out_rows: int, *, k_out=None, v_out=None,
            stream=None):
    """stepkv_compact: dense retained cache [L][Hkv][out_rows][d] for K and V."""
    import torch

    lib = load()
    L, Hkv, d, dev = pb.num_layers, pb.num_kv_heads, pb.head_dim, pb.device
    kp = _need(k, torch.bfloat16, (L, Hkv, pb.ntot, d), "k")
    vp = _need(v, torch.bfloat16, (L, Hkv, pb.ntot, d), "v")
    ip = _need(idx, torch.int32, (L, Hkv, pb.ntot), "idx")
    cp = _need(cu_retained, torch.int32, (pb.num_seqs + 1,), "cu_retained")
    if k_out is None:
        k_out = torch.empty((L, Hkv, out_rows, d), dtype=torch.bfloat16, device=dev)
    if v_out is None:
        v_out = torch.empty((L, Hkv, out_rows, d), dtype=torch.bfloat16, device=dev)
    _need(k_out, torch.bfloat16, (L, Hkv, out_rows, d), "k_out")
    _need(v_out, torch.bfloat16, (L, Hkv, out_rows, d), "v_out")
    rc = lib.stepkv_compact(ctypes.byref(pb.c), kp, vp, ip, cp, int(out_rows), k_out.data_ptr(),
                            v_out.data_ptr(), _stream(stream))
    _check("stepkv_compact", rc)
    return k_out, v_out


def decode_attention(pb: Problem, q_dec, k_hat, v_hat, cu_retained, out_rows: int,
                     scale: float = 0.0, *, workspace=None, out=None, stream=None):
    """stepkv_decode_attention: fp32 [L][S][Hq][d]."""
    import torch

    lib = load()
    L, S, Hq, Hkv, d = pb.num_layers, pb.num_seqs, pb.num_q_heads, pb.num_kv_heads, pb.head_dim
    qp = _need(q_dec, torch.bfloat16, (L, S, Hq, d), "q_dec")
    kp = _need(k_hat, torch.bfloat16, (L, Hkv, out_rows, d), "k_hat")
    vp = _need(v_hat, torch.bfloat16, (L, Hkv, out_rows, d), "v_hat")
    cp = _need(cu_retained, torch.int32, (S + 1,), "cu_retained")
    if out is None:
        out = torch.empty((L, S, Hq, d), dtype=torch.float32, device=pb.device)
    _need(out, torch.float32, (L, S, Hq, d), "out")
    if workspace is None:
        need = int(lib.stepkv_decode_workspace_bytes(ctypes.byref(pb.c), int(out_rows)))
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=pb.device)
    rc = lib.stepkv_decode_attention(ctypes.byref(pb.c), qp, kp, vp, cp, int(out_rows),
                                     float(scale), out.data_ptr(), workspace.data_ptr(),
                                     workspace.numel(), _stream(stream))
    _check("stepkv_decode_attention", rc)
    return out


def retained_rows(pb: Problem, protected, budget: int, budgets=None) -> np.ndarray:
    """stepkv_retained_rows (host): cu_retained [S+1] int32 of the compacted cache, from the
    host protected mask uint8 [Ntot] and the budget (or per-sequence budgets [S])."""
    prot = np.ascontiguousarray(protected, dtype=np.uint8)
    if prot.shape != (pb.ntot,):
        raise ValueError(f"protected: shape {prot.shape}, expected ({pb.ntot},)")
    bud = None if budgets is None else np.ascontiguousarray(budgets, dtype=np.int32)
    if bud is not None and bud.shape != (pb.num_seqs,):
        raise ValueError(f"budgets: shape {bud.shape}, expected ({pb.num_seqs},)")
    cu = np.zeros(pb.num_seqs + 1, np.int32)
    rc = load().stepkv_retained_rows(ctypes.byref(pb.c), prot.ctypes.data, int(budget),
                                     bud.ctypes.data if bud is not None else None, cu.ctypes.data)
    _check("stepkv_retained_rows", rc)
    return cu


def compress(pb: Problem, q_win, k, v, step_ids, protected, step_utility, budget: int,
             out_rows: int, params: Optional[Params] = None, *, lse=None, budgets=None,
             scores=None, idx=None, cu_retained=None, k_out=None, v_out=None, workspace=None,
             stream=None):
    """stepkv_compress: score -> select -> compact in one library call on one stream.

    Returns scores [L][Hkv][Ntot], idx [L][Hkv][Ntot], cu_retained [S+1] and the compacted
    k_hat / v_hat [L][Hkv][out_rows][d]. With `lse` the saliency takes one sweep."""
    import torch

    lib = load()
    L, Hkv, d, W, S, dev = (pb.num_layers, pb.num_kv_heads, pb.head_dim, pb.window, pb.num_seqs,
                            pb.device)
    qp = _need(q_win, torch.bfloat16, (L, S, W, pb.num_q_heads, d), "q_win")
    kp = _need(k, torch.bfloat16, (L, Hkv, pb.ntot, d), "k")
    vp = _need(v, torch.bfloat16, (L, Hkv, pb.ntot, d), "v")
    lp = _need(lse, torch.float32, (L, S, W, pb.num_q_heads), "lse") if lse is not None else None
    sp = _need(step_ids, torch.int32, (pb.ntot,), "step_ids")
    pp = _need(protected, torch.uint8, (pb.ntot,), "protected")
    up = _need(step_utility, torch.float32, (pb.total_steps,), "step_utility")
    bp = _need(budgets, torch.int32, (S,), "budgets") if budgets is not None else None
    if scores is None:
        scores = torch.empty((L, Hkv, pb.ntot), dtype=torch.float32, device=dev)
    if idx is None:
        idx = torch.empty((L, Hkv, pb.ntot), dtype=torch.int32, device=dev)
    if cu_retained is None:
        cu_retained = torch.empty(S + 1, dtype=torch.int32, device=dev)
    if k_out is None:
        k_out = torch.empty((L, Hkv, out_rows, d), dtype=torch.bfloat16, device=dev)
    if v_out is None:
        v_out = torch.empty((L, Hkv, out_rows, d), dtype=torch.bfloat16, device=dev)
    for t, dt, shape, name in ((scores, torch.float32, (L, Hkv, pb.ntot), "scores"),
                               (idx, torch.int32, (L, Hkv, pb.ntot), "idx"),
                               (cu_retained, torch.int32, (S + 1,), "cu_retained"),
                               (k_out, torch.bfloat16, (L, Hkv, out_rows, d), "k_out"),
                               (v_out, torch.bfloat16, (L, Hkv, out_rows, d), "v_out")):
        _need(t, dt, shape, name)
    if workspace is None:
        need = int(lib.stepkv_compress_workspace_bytes(ctypes.byref(pb.c)))
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    rc = lib.stepkv_compress(ctypes.byref(pb.c), ctypes.byref((params or Params()).c()), qp, kp,
                             vp, lp, sp, pp, up, int(budget), bp, scores.data_ptr(),
                             idx.data_ptr(), cu_retained.data_ptr(), int(out_rows),
                             k_out.data_ptr(), v_out.data_ptr(), workspace.data_ptr(),
                             workspace.numel(), _stream(stream))
    _check("stepkv_compress", rc)
    return {"scores": scores, "idx": idx, "cu_retained": cu_retained, "k_hat": k_out,
            "v_hat": v_out}


def bandwidth_probe(src, dst, copy: bool, stream=None) -> None:
    """stepkv_bandwidth_probe: read src (copy False) or copy src to dst, with the
    compaction's access width; both contiguous CUDA tensors, src.nbytes a multiple of 16."""
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < (nbytes if copy else 4 * ((nbytes // 16 + 255) // 256)):
        raise ValueError("dst too small")
    _check("stepkv_bandwidth_probe", load().stepkv_bandwidth_probe(
        src.data_ptr(), dst.data_ptr(), nbytes, int(bool(copy)), _stream(stream)))


def issue_probe(mix: bool, blocks: int, iters: int, sink, stream=None) -> None:
    """stepkv_issue_probe: four 32x32x16 bf16 MFMAs per loop per wave, alone (mix False) or
    with the saliency sweeps' vector work for two score elements per MFMA; sink a float32
    CUDA tensor of at least blocks * 256 elements."""
    if sink.numel() < blocks * 256 or sink.dtype.itemsize != 4:
        raise ValueError("sink too small")
    _check("stepkv_issue_probe", load().stepkv_issue_probe(int(bool(mix)), int(blocks), int(iters),
                                                           sink.data_ptr(), _stream(stream)))


def bf16_from_bits(bits: np.ndarray, device="cuda"):
    """Move bf16 bit patterns (uint16 numpy) to a torch bfloat16 tensor on `device`."""
    import torch

    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(
        torch.bfloat16)
