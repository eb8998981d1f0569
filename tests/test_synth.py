"""Input generator checks: determinism, shapes and the step-span structure."""
import math

import numpy as np
import pytest

from synth import bf16_bits_to_f32, f32_to_bf16_bits, make_workload


def test_bf16_round_to_nearest_even():
    one = 1.0
    x = np.array([one, one + 2**-8, one + 3 * 2**-8, one + 2**-8 + 2**-20, -2.5, 0.0, -0.0],
                 dtype=np.float32)
    b = f32_to_bf16_bits(x)
    assert list(b) == [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC020, 0x0000, 0x8000]
    assert (bf16_bits_to_f32(b)[[0, 4]] == np.array([1.0, -2.5], np.float32)).all()


def test_deterministic_per_seed():
    a = make_workload("tiny", 233)
    b = make_workload("tiny", 233)
    c = make_workload("tiny", 42)
    for f in ("q_win", "k", "v", "step_ids", "protected"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    assert not np.array_equal(a.k, c.k)
    assert all(np.array_equal(x.obs_sim, y.obs_sim) for x, y in zip(a.signals, b.signals))


def _check_steps(w):
    for s in range(w.num_seqs):
        a, b = int(w.cu_seqlens[s]), int(w.cu_seqlens[s + 1])
        p = w.protected_len[s]
        assert (w.protected[a:a + p] == 1).all() and (w.protected[a + p:b] == 0).all()
        assert (w.step_ids[a:a + p] == -1).all()
        sid = w.step_ids[a + p:b]
        n = int(w.cu_steps[s + 1] - w.cu_steps[s])
        assert sid[0] == 0 and sid[-1] == n - 1
        assert (np.diff(sid) >= 0).all() and (np.diff(sid) <= 1).all()  # contiguous spans
        assert w.signals[s].num_steps == n
        assert w.signals[s].gain[0] == 1.0 and w.signals[s].red[0] == 0.0


def test_tiny_shapes():
    w = make_workload("tiny")
    assert w.q_win.shape == (1, 1, 32, 4, 64)
    assert w.k.shape == w.v.shape == (1, 2, 1024, 64)
    assert w.cu_steps[-1] == 8 and w.budget == 128 and w.pool_kernel == 7
    _check_steps(w)
    std = bf16_bits_to_f32(w.k).std()
    assert abs(std - 1 / 8) < 0.01


def test_l1_8k_outlier_channels():
    w = make_workload("l1_8k")
    assert w.k.shape == (1, 8, 8192, 128) and w.cu_steps[-1] == 24
    _check_steps(w)
    kf = bf16_bits_to_f32(w.k[0, 3])
    ch_std = kf.std(axis=0)
    big = np.sort(ch_std)[-4:]
    assert (big > 0.6).all() and np.sort(ch_std)[-5] < 0.15  # four channels at 8/sqrt(128)


def test_l32_32k_structure_one_layer():
    w = make_workload("l32_32k", num_layers=1, with_v=False)
    assert w.q_win.shape == (1, 1, 64, 32, 128)
    assert w.cu_steps[-1] == 96 and w.seqlens == [32768] and w.protected_len == [512]
    _check_steps(w)
    lens = np.bincount(w.step_ids[w.step_ids >= 0])
    assert lens.max() <= 2048 and lens.sum() == 32768 - 512
    planted = w.planted_steps[0]
    assert len(planted) == 5 and max(planted) < 32
    # planted steps are reused by later observations: sim drawn from U(0.5, 1)
    sim = w.signals[0].obs_sim
    for k in planted:
        assert (sim[k + 1:, k] >= 0.5).all()


def test_ragged16_structure():
    w = make_workload("ragged16", num_layers=1, with_v=False)
    assert w.num_seqs == 16 and w.k.shape[:2] == (1, 4) and w.q_dec.shape == (1, 16, 28, 128)
    assert all(4096 <= n <= 32768 for n in w.seqlens)
    steps = np.diff(w.cu_steps)
    assert steps.min() >= 12 and steps.max() <= 80
    _check_steps(w)


@pytest.mark.parametrize("name", ["l32_16k", "l32_32k", "ragged16"])
def test_reduced_sizes_keep_structure(name):
    w = make_workload(name, seqlens=[3001, 1500][: (2 if name == "ragged16" else 1)],
                      num_layers=2, num_steps=12)
    _check_steps(w)
    assert w.k.shape[0] == 2
