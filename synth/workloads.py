"""Seeded generators for agent-trajectory-shaped KV caches.

Every array is produced on the host with numpy's PCG64, from a seed and a
configuration name, so the HIP path and the CPU oracle can be fed the very
same bits. Nothing here computes saliency, step utility, priorities or a
selection: the per-step signals (validity, evidence gain, action redundancy,
observation similarity) are drawn at random and handed over raw.

Layouts (bf16 values are stored as their uint16 bit patterns):

* ``q_win``  uint16 ``[L][S][W][Hq][d]``  the last W queries of every sequence
* ``k``, ``v`` uint16 ``[L][Hkv][Ntot][d]`` sequences concatenated along Ntot
* ``step_ids`` int32 ``[Ntot]``  step index local to its sequence, -1 if protected
* ``protected`` uint8 ``[Ntot]``  1 for the protected prompt/query prefix
* ``cu_seqlens`` int32 ``[S+1]``, ``cu_steps`` int32 ``[S+1]``
* ``q_dec`` uint16 ``[L][S][Hq][d]`` one decode query per sequence (ragged case)

Normal draws use a 65536-entry inverse-CDF quantile table indexed by 16-bit
uniform words (a discretised N(0,1), exact to the bf16 grid it is rounded to,
with tails truncated at about 4.3 sigma). It is several times faster than
numpy's ziggurat sampler, which matters for the 2-8 GiB caches.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence

import numpy as np

SEEDS = (233, 42, 3407)  # the three seeds the paper's experiments use (App. D)

CONFIG_NAMES = ("tiny", "l1_8k", "l32_16k", "l32_32k", "ragged16")

_QUANTILES: Optional[np.ndarray] = None
_TABLES: Dict[float, np.ndarray] = {}


# ----------------------------------------------------------------- bf16 bits
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); return bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = u + np.uint32(0x7FFF)
    r += (u >> np.uint32(16)) & np.uint32(1)
    return (r >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Decode bf16 bit patterns to float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal_table(scale: float) -> np.ndarray:
    """bf16 bits of scale * Phi^-1((j + 1/2) / 65536) for j in [0, 65536)."""
    global _QUANTILES
    if _QUANTILES is None:
        from scipy.special import ndtri

        _QUANTILES = ndtri((np.arange(65536, dtype=np.float64) + 0.5) / 65536.0)
    key = float(scale)
    if key not in _TABLES:
        _TABLES[key] = f32_to_bf16_bits((_QUANTILES * key).astype(np.float32))
    return _TABLES[key]


def _fill_normal_bf16(bitgen: np.random.PCG64, out: np.ndarray, scale: float) -> None:
    """Fill a uint16 array with bf16 bits of N(0, scale^2) draws, in 4 Mi blocks."""
    tab = _normal_table(scale)
    flat = out.reshape(-1)
    block = 1 << 22
    for s in range(0, flat.size, block):
        n = min(block, flat.size - s)
        words = bitgen.random_raw((n + 3) // 4).view(np.uint16)[:n]
        np.take(tab, words, out=flat[s:s + n])


def _fill_slabs(seed: np.random.SeedSequence, out: np.ndarray, scale: float) -> None:
    """Fill out[i] for every leading index i from its own spawned stream.

    Each slab has an independent PCG64 stream, so the result does not depend
    on how many threads share the work (numpy releases the GIL in both the raw
    draw and the table gather).
    """
    _normal_table(scale)  # build the table once, outside the threads
    kids = seed.spawn(out.shape[0])

    def one(i: int) -> None:
        _fill_normal_bf16(np.random.PCG64(kids[i]), out[i], scale)

    workers = max(1, min(16, os.cpu_count() or 1, out.shape[0]))
    if workers == 1:
        for i in range(out.shape[0]):
            one(i)
        return
    with ThreadPoolExecutor(workers) as ex:
        list(ex.map(one, range(out.shape[0])))


# ---------------------------------------------------------------- containers
@dataclasses.dataclass
class StepSignals:
    """Raw per-step signals of one trajectory (inputs to the step-utility update).

    ``obs_sim[t, k]`` (k < t) is the similarity of observation t to observation k
    seen at boundary t; entries on and above the diagonal are unused zeros.
    """

    valid: np.ndarray  # float32 [n] in {0, 1}
    gain: np.ndarray  # float32 [n] in [0, 1], gain[0] = 1
    red: np.ndarray  # float32 [n] in [0, 1], red[0] = 0
    obs_sim: np.ndarray  # float32 [n, n]

    @property
    def num_steps(self) -> int:
        return int(self.valid.shape[0])


@dataclasses.dataclass
class Workload:
    name: str
    seed: int
    num_layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    window: int
    pool_kernel: int
    budget: int
    seqlens: List[int]
    protected_len: List[int]
    cu_seqlens: np.ndarray
    cu_steps: np.ndarray
    step_ids: np.ndarray
    protected: np.ndarray
    signals: List[StepSignals]
    q_win: np.ndarray
    k: np.ndarray
    v: np.ndarray
    q_dec: Optional[np.ndarray] = None
    planted_steps: Optional[List[List[int]]] = None

    @property
    def num_seqs(self) -> int:
        return len(self.seqlens)

    @property
    def total_tokens(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def total_steps(self) -> int:
        return int(self.cu_steps[-1])


# ------------------------------------------------------------ step spans
def _integerise(x: np.ndarray, total: int, cap: Optional[int] = None) -> np.ndarray:
    """Integer lengths >= 1 (and <= cap) summing to ``total``, closest to x."""
    n = x.shape[0]
    if total < n:
        raise ValueError("fewer tokens than steps")
    base = np.maximum(np.floor(x).astype(np.int64), 1)
    if cap is not None:
        base = np.minimum(base, cap)
    frac = x - np.floor(x)
    diff = total - int(base.sum())
    order = np.argsort(-frac, kind="stable")
    i = 0
    guard = 0
    while diff != 0:
        j = order[i % n]
        if diff > 0 and (cap is None or base[j] < cap):
            base[j] += 1
            diff -= 1
        elif diff < 0 and base[j] > 1:
            base[j] -= 1
            diff += 1
        i += 1
        guard += 1
        if guard > 64 * n + 4 * abs(total):
            raise RuntimeError("cannot integerise step lengths")
    return base


def _rescale(x: np.ndarray, total: int) -> np.ndarray:
    return _integerise(x * (total / x.sum()), total)


def _spans_uniform_truncated(rng, n, lo, hi, total):
    """n lengths ~ U{lo..hi}; the last step is padded or truncated to fill total.

    Draws are repeated until the first n-1 steps leave at least one token.
    """
    n = min(n, total)
    for _ in range(1000):
        lens = rng.integers(lo, hi + 1, size=n).astype(np.int64)
        head = int(lens[:-1].sum())
        if head <= total - 1:
            lens[-1] = total - head
            return lens
    return _rescale(np.ones(n), total)


def _spans_lognormal(rng, n, mu, sigma, total):
    n = min(n, total)
    return _rescale(rng.lognormal(mu, sigma, size=n), total)


def _spans_alternating(rng, n, total, short=(32, 128), long_mean=600.0, sigma=0.6):
    """Alternating short thought/action and long observation segments."""
    n = min(n, total)
    mu = math.log(long_mean) - 0.5 * sigma * sigma
    x = np.empty(n, dtype=np.float64)
    for i in range(n):
        if i % 2 == 0:
            x[i] = rng.integers(short[0], short[1] + 1)
        else:
            x[i] = rng.lognormal(mu, sigma)
    return _rescale(x, total)


def _spans_pareto(rng, n, alpha, cap, total):
    """Pareto(alpha) lengths x_m * (1 + Lomax), capped, x_m bisected to hit total."""
    n = min(n, total)
    u = 1.0 + rng.pareto(alpha, size=n)
    if n * cap < total:
        raise ValueError("cap too small for total")
    lo, hi = 0.0, float(cap) * 4.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if np.minimum(cap, mid * u).sum() < total:
            lo = mid
        else:
            hi = mid
    return _integerise(np.minimum(cap, hi * u), total, cap=cap)


# ------------------------------------------------------------ step signals
def _signals(rng, n, planted: Sequence[int] = ()) -> StepSignals:
    valid = (rng.random(n) < 0.8).astype(np.float32)
    gain = rng.random(n).astype(np.float32)
    red = rng.random(n).astype(np.float32)
    gain[0] = 1.0
    red[0] = 0.0
    sim = np.zeros((n, n), dtype=np.float32)
    for t in range(1, n):
        hit = rng.random(t) < 0.2
        sim[t, :t] = np.where(hit, rng.random(t), 0.0)
        for k in planted:
            if k < t:
                sim[t, k] = rng.uniform(0.5, 1.0)
    return StepSignals(valid=valid, gain=gain, red=red, obs_sim=sim)


# ------------------------------------------------------------ configurations
_BASE = {
    # 1 layer, GQA 4/2, d 64, N 1024, 8 uniform steps, 64 protected, W 32, B 128
    "tiny": dict(L=1, Hq=4, Hkv=2, d=64, W=32, B=128, pool=7, seqlens=[1024], prot=64,
                 steps="uniform8"),
    # Llama-3-8B single layer, N 8192, 24 lognormal steps, 256 protected, W 32, B 512
    "l1_8k": dict(L=1, Hq=32, Hkv=8, d=128, W=32, B=512, pool=7, seqlens=[8192], prot=256,
                  steps="lognormal24", outliers=4),
    # 32 layers, N 16384, 48 alternating steps, 512 protected, W 32, B 1024
    "l32_16k": dict(L=32, Hq=32, Hkv=8, d=128, W=32, B=1024, pool=7, seqlens=[16384],
                    prot=512, steps="alternating48"),
    # 32 layers, N 32768, 96 Pareto steps, planted rank-8 keys, W 64, B 1024
    "l32_32k": dict(L=32, Hq=32, Hkv=8, d=128, W=64, B=1024, pool=7, seqlens=[32768],
                    prot=512, steps="pareto96", planted=5),
    # Qwen2.5-7B-like ragged batch of 16, 28 layers, G 7, W 32, B 2048
    "ragged16": dict(L=28, Hq=28, Hkv=4, d=128, W=32, B=2048, pool=7, seqlens="ragged16",
                     prot=512, steps="alternating_rand", decode=True),
}


def make_workload(
    name: str,
    seed: int = 233,
    *,
    seqlens: Optional[Sequence[int]] = None,
    num_layers: Optional[int] = None,
    window: Optional[int] = None,
    budget: Optional[int] = None,
    protected_len: Optional[int] = None,
    num_steps: Optional[int] = None,
    with_v: bool = True,
) -> Workload:
    """Build one seeded workload; keyword overrides shrink it for parity tests.

    The overrides keep every structural rule of the named configuration
    (step-length law, planted keys, outlier channels, GQA shape) and only
    change the sizes.
    """
    if name not in _BASE:
        raise KeyError(f"unknown workload {name!r}; choose from {CONFIG_NAMES}")
    cfg = dict(_BASE[name])
    ss = np.random.SeedSequence([seed, CONFIG_NAMES.index(name)])
    s_struct, s_q, s_k, s_v, s_plant, s_dec = ss.spawn(6)
    rng = np.random.Generator(np.random.PCG64(s_struct))

    L = num_layers if num_layers is not None else cfg["L"]
    Hq, Hkv, d = cfg["Hq"], cfg["Hkv"], cfg["d"]
    W = window if window is not None else cfg["W"]
    B = budget if budget is not None else cfg["B"]

    if seqlens is None:
        if cfg["seqlens"] == "ragged16":
            seqlens = [int(x) for x in rng.integers(4096, 32768 + 1, size=16)]
        else:
            seqlens = list(cfg["seqlens"])
    seqlens = [int(n) for n in seqlens]
    S = len(seqlens)
    if protected_len is None:
        protected_len = cfg["prot"]
    prot = [min(int(protected_len), n) for n in seqlens]

    # step spans tile [prot, N) of every sequence
    spans: List[np.ndarray] = []
    for s in range(S):
        total = seqlens[s] - prot[s]
        kind = cfg["steps"]
        if total <= 0:
            spans.append(np.zeros(0, dtype=np.int64))
            continue
        if kind == "uniform8":
            lens = _spans_uniform_truncated(rng, num_steps or 8, 64, 192, total)
        elif kind == "lognormal24":
            lens = _spans_lognormal(rng, num_steps or 24, 5.5, 0.6, total)
        elif kind == "alternating48":
            lens = _spans_alternating(rng, num_steps or 48, total)
        elif kind == "pareto96":
            lens = _spans_pareto(rng, num_steps or 96, 1.5, 2048, total)
        elif kind == "alternating_rand":
            n = num_steps or int(rng.integers(12, 80 + 1))
            lens = _spans_alternating(rng, n, total)
        else:  # pragma: no cover
            raise AssertionError(kind)
        spans.append(lens)

    cu_seqlens = np.zeros(S + 1, dtype=np.int32)
    cu_seqlens[1:] = np.cumsum(seqlens)
    ntot = int(cu_seqlens[-1])
    cu_steps = np.zeros(S + 1, dtype=np.int32)
    cu_steps[1:] = np.cumsum([len(x) for x in spans])
    step_ids = np.full(ntot, -1, dtype=np.int32)
    protected = np.zeros(ntot, dtype=np.uint8)
    planted_steps: List[List[int]] = []
    signals: List[StepSignals] = []
    for s in range(S):
        base = int(cu_seqlens[s])
        protected[base:base + prot[s]] = 1
        pos = base + prot[s]
        for k, ln in enumerate(spans[s]):
            step_ids[pos:pos + int(ln)] = k
            pos += int(ln)
        n = len(spans[s])
        planted: List[int] = []
        if cfg.get("planted") and n > 0:
            early = max(1, n // 3)
            planted = sorted(int(x) for x in rng.choice(early, size=min(cfg["planted"], early),
                                                         replace=False))
        planted_steps.append(planted)
        signals.append(_signals(rng, n, planted) if n > 0 else
                       StepSignals(*(np.zeros(0, np.float32),) * 3, np.zeros((0, 0), np.float32)))

    # observation-window queries N(0,1), keys/values N(0,1)/sqrt(d)
    q_win = np.empty((L, S, W, Hq, d), dtype=np.uint16)
    _fill_slabs(s_q, q_win, 1.0)
    k = np.empty((L, Hkv, ntot, d), dtype=np.uint16)
    _fill_slabs(s_k, k.reshape(L * Hkv, ntot, d), 1.0 / math.sqrt(d))
    if with_v:
        v = np.empty((L, Hkv, ntot, d), dtype=np.uint16)
        _fill_slabs(s_v, v.reshape(L * Hkv, ntot, d), 1.0 / math.sqrt(d))
    else:
        v = np.zeros((0,), dtype=np.uint16)

    prng = np.random.Generator(np.random.PCG64(s_plant))
    if cfg.get("outliers"):
        # a few key channels per head carry 8x the magnitude (exact in bf16)
        for l in range(L):
            for h in range(Hkv):
                ch = prng.choice(d, size=cfg["outliers"], replace=False)
                blk = bf16_bits_to_f32(k[l, h][:, ch]) * np.float32(8.0)
                k[l, h][:, ch] = f32_to_bf16_bits(blk)
    if cfg.get("planted"):
        # rank-8 component shared by the planted early steps; window rows align
        # with it so those keys gain about 2 nats of logit (kappa*gamma/sqrt(d)=2)
        kappa, gamma = math.sqrt(d), 2.0
        G = Hq // Hkv
        for s in range(S):
            if not planted_steps[s]:
                continue
            base = int(cu_seqlens[s])
            loc = np.nonzero(np.isin(step_ids[base:base + seqlens[s]], planted_steps[s]))[0]
            rows = base + loc
            for l in range(L):
                for h in range(Hkv):
                    U, _ = np.linalg.qr(prng.standard_normal((d, 8)))
                    a = prng.standard_normal(8)
                    a /= np.linalg.norm(a)
                    eps = prng.standard_normal((rows.size, 8)) * (0.3 / math.sqrt(8))
                    kf = bf16_bits_to_f32(k[l, h, rows]).astype(np.float64)
                    kf += kappa * (a + eps) @ U.T
                    k[l, h, rows] = f32_to_bf16_bits(kf.astype(np.float32))
                    dl = prng.standard_normal((W, G, 8)) * (0.3 / math.sqrt(8))
                    qf = bf16_bits_to_f32(q_win[l, s, :, h * G:(h + 1) * G]).astype(np.float64)
                    qf += gamma * (a + dl) @ U.T
                    q_win[l, s, :, h * G:(h + 1) * G] = f32_to_bf16_bits(qf.astype(np.float32))

    q_dec = None
    if cfg.get("decode"):
        q_dec = np.empty((L, S, Hq, d), dtype=np.uint16)
        _fill_slabs(s_dec, q_dec, 1.0)

    return Workload(
        name=name, seed=seed, num_layers=L, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d,
        window=W, pool_kernel=cfg["pool"], budget=B, seqlens=seqlens, protected_len=prot,
        cu_seqlens=cu_seqlens, cu_steps=cu_steps, step_ids=step_ids, protected=protected,
        signals=signals, q_win=q_win, k=k, v=v, q_dec=q_dec, planted_steps=planted_steps,
    )
