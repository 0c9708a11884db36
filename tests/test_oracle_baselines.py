"""Pins of the oracle's critic-free baselines: GRPO's group normalisation (Sec. 2) and the
running-mean reward window (Sec. 4.3, Sec. 4.5)."""
import math

import numpy as np
import pytest

from oracle import group_advantage, running_mean_advantage, trajectory_rewards
from synth import generate, small_config


def _one_token_trajectories(R, mask=None):
    B = len(R)
    return (np.asarray(R, np.float32), np.ones(B, np.uint8) if mask is None else np.asarray(mask, np.uint8),
            np.arange(B + 1, dtype=np.int32))


def test_grpo_hand_worked_group():
    # One group of four with rewards (1, 0, 0, 1): mu = 0.5, variance 0.25, sigma = 0.5 at
    # eps = 0, so A = (1, -1, -1, 1); with eps = 0.75 sigma = 1 and A = (0.5, -0.5, -0.5, 0.5).
    r, m, cu = _one_token_trajectories([1, 0, 0, 1])
    adv, A, R, n = group_advantage(r, m, cu, 4, 0.0)
    assert A.tolist() == [1, -1, -1, 1] and adv.tolist() == [1, -1, -1, 1] and n == 4
    assert group_advantage(r, m, cu, 4, 0.75)[1].tolist() == [0.5, -0.5, -0.5, 0.5]
    # two groups of two are normalised separately
    assert group_advantage(r, m, cu, 2, 0.0)[1].tolist() == [1, -1, -1, 1]


def test_grpo_moments_and_invariance():
    rng = np.random.default_rng(5)
    R = rng.normal(0.3, 1.7, 64)
    r, m, cu = _one_token_trajectories(R)
    for G in (4, 8, 16):
        _, A, Rb, _ = group_advantage(r, m, cu, G, 1e-6)
        g = A.reshape(-1, G)
        var = np.var(Rb.reshape(-1, G), axis=1)
        assert np.allclose(g.mean(axis=1), 0.0, atol=1e-12)                     # centred
        assert np.allclose((g ** 2).mean(axis=1), var / (var + 1e-6), rtol=1e-12)  # scaled
        # with eps = 0, a positive affine change of the rewards leaves A unchanged
        _, A0, _, _ = group_advantage(r, m, cu, G, 0.0)
        _, A1, _, _ = group_advantage((3.0 * r.astype(np.float64) + 2.0), m, cu, G, 0.0)
        assert np.allclose(A0, A1, rtol=1e-12, atol=1e-12)


def test_grpo_equal_rewards_and_token_broadcast():
    r, m, cu = _one_token_trajectories([2, 2, 2, 2])
    assert group_advantage(r, m, cu, 4, 1e-4)[1].tolist() == [0, 0, 0, 0]
    assert all(math.isnan(a) for a in group_advantage(r, m, cu, 4, 0.0)[1])   # 0/0, as printed
    b = generate(small_config("g1", 121, B=8, T=2000, H=8, V=8))
    adv, A, R, n = group_advantage(b.rewards, b.mask, b.cu_seqlens, 4, 1e-6)
    assert np.array_equal(R, trajectory_rewards(b.rewards, b.cu_seqlens))
    for i in range(8):
        s, e = b.cu_seqlens[i], b.cu_seqlens[i + 1]
        seg = adv[s:e]
        assert (seg[b.mask[s:e] == 1] == A[i]).all() and (seg[b.mask[s:e] == 0] == 0).all()


def test_running_mean_hand_worked_window():
    # Window 3 after history (1, 0); batch rewards (1, 1, 0, 0):
    #   b0: mean(1, 0) = 1/2, b1: mean(1, 0, 1) = 2/3, b2: mean(0, 1, 1) = 2/3, b3: mean(1, 1, 0) = 2/3
    r, m, cu = _one_token_trajectories([1, 1, 0, 0])
    _, A, _, _, hist = running_mean_advantage(r, m, cu, 3, {0: [1.0, 0.0]})
    assert A == pytest.approx([0.5, 1 / 3, -2 / 3, -2 / 3], rel=1e-15)
    assert hist[0] == [1.0, 0.0, 1.0, 1.0, 0.0, 0.0]


def test_running_mean_empty_window_keys_and_long_window():
    r, m, cu = _one_token_trajectories([0.5, 2.0, 1.0])
    _, A, _, _, _ = running_mean_advantage(r, m, cu, 8)
    assert A.tolist() == [0.5, 2.0 - 0.5, 1.0 - 1.25]          # empty window: baseline 0
    # keyed windows equal separate runs per key
    rng = np.random.default_rng(6)
    R = rng.random(40)
    keys = rng.integers(0, 3, 40)
    r, m, cu = _one_token_trajectories(R)
    hist = {0: [0.25], 2: [1.0, 0.0]}
    _, A, _, _, h2 = running_mean_advantage(r, m, cu, 4, hist, keys)
    for k in range(3):
        idx = np.nonzero(keys == k)[0]
        rk, mk, ck = _one_token_trajectories(R[idx])
        _, Ak, _, _, hk = running_mean_advantage(rk, mk, ck, 4, {0: hist.get(k, [])})
        assert np.array_equal(A[idx], Ak) and h2[k] == hk[0]
    # a window longer than the whole past is the cumulative mean of everything before
    r, m, cu = _one_token_trajectories(R)
    _, A, _, _, _ = running_mean_advantage(r, m, cu, 1000, {0: [0.0, 1.0]})
    past = np.concatenate([[0.0, 1.0], R.astype(np.float32).astype(np.float64)])
    cum = np.array([past[:2 + i].mean() for i in range(40)])
    assert np.allclose(A, R.astype(np.float32) - cum, rtol=1e-13, atol=1e-15)
