"""Pins of the oracle's skip-observation GAE (Sec. 3.2, Eq. 4-5) and returns."""
import math

import numpy as np
import pytest

from oracle import advantage
from oracle.sao_oracle import trajectory_lambda
from synth import CONFIGS, generate
from tests.golden.load import gae_example


def textbook_gae(values, rewards, gamma, lam):
    """Sec. 2 GAE as the explicit sum A_t = sum_l (gamma lam)^l delta_{t+l} (model tokens only)."""
    v = [float(x) for x in values] + [0.0]
    n = len(rewards)
    delta = [float(rewards[t]) + gamma * v[t + 1] - v[t] for t in range(n)]
    return np.array([math.fsum((gamma * lam) ** l * delta[t + l] for l in range(n - t))
                     for t in range(n)])


def _traj(seed, n, p_obs=0.0, dense=False):
    rng = np.random.default_rng(seed)
    vals = rng.normal(0.5, 0.2, n).astype(np.float32)
    rew = np.zeros(n, np.float32)
    if dense:
        rew[:] = rng.normal(0, 1, n)
    rew[-1] = 1.0
    mask = (rng.random(n) >= p_obs).astype(np.uint8)
    mask[-1] = 1
    return vals, rew, mask


def test_golden_worked_example():
    ex = gae_example()
    adv, ret, N = advantage(ex["values"], ex["rewards"], ex["mask"], ex["cu"], ex["gamma"],
                            ex["lam"], alpha=0.0)
    assert N == int(ex["mask"].sum())
    assert np.allclose(adv, ex["adv"], atol=1e-6, rtol=0)
    assert np.allclose(ret, ex["ret"], atol=1e-6, rtol=0)


@pytest.mark.parametrize("gamma,lam", [(1.0, 1.0), (0.99, 0.95), (0.9, 0.5), (1.0, 0.0)])
def test_no_observations_is_textbook_gae(gamma, lam):
    vals, rew, _ = _traj(10, 57, dense=True)
    mask = np.ones(57, np.uint8)
    adv, _, _ = advantage(vals, rew, mask, np.array([0, 57]), gamma, lam)
    assert np.allclose(adv, textbook_gae(vals, rew, gamma, lam), rtol=1e-12, atol=1e-12)


def test_lambda_gamma_one_is_return_minus_value():
    b = generate(CONFIGS["c1"], with_head=False)
    adv, ret, _ = advantage(b.values, b.rewards, b.mask, b.cu_seqlens, 1.0, 1.0, alpha=0.0)
    m = b.mask == 1
    assert np.allclose(adv[m], ret[m] - b.values[m].astype(np.float64), rtol=0, atol=1e-9)
    # one terminal reward R per trajectory: A_t = R - V_t
    for i in range(b.cfg.B):
        s, e = b.cu_seqlens[i], b.cu_seqlens[i + 1]
        R = float(b.rewards[e - 1])
        mm = b.mask[s:e] == 1
        assert np.allclose(adv[s:e][mm], R - b.values[s:e][mm].astype(np.float64), atol=1e-9)


def test_lambda_zero_is_td_residual_and_gamma_zero():
    vals, rew, mask = _traj(11, 40, p_obs=0.0, dense=True)
    adv, _, _ = advantage(vals, rew, mask, np.array([0, 40]), 0.97, 0.0)
    v_next = np.append(vals[1:].astype(np.float64), 0.0)
    assert np.allclose(adv, rew + 0.97 * v_next - vals, atol=1e-12)
    adv0, ret0, _ = advantage(vals, rew, mask, np.array([0, 40]), 0.0, 0.7)
    assert np.allclose(adv0, rew.astype(np.float64) - vals, atol=1e-12)
    assert np.allclose(ret0, rew, atol=1e-12)


def test_deleting_observations_changes_nothing():
    vals, rew, mask = _traj(12, 300, p_obs=0.35)
    rew[mask == 0] = 0.0
    cu = np.array([0, 300])
    adv, ret, _ = advantage(vals, rew, mask, cu, 0.99, 0.9)
    keep = mask == 1
    adv2, ret2, _ = advantage(vals[keep], rew[keep], mask[keep], np.array([0, keep.sum()]), 0.99, 0.9)
    assert np.array_equal(adv[keep], adv2) and np.array_equal(ret[keep], ret2)
    assert (adv[~keep] == 0).all() and (ret[~keep] == 0).all()


def test_observation_reward_folds_into_preceding_action():
    vals, rew, mask = _traj(13, 120, p_obs=0.4)
    rew[:] = 0.0
    obs = np.nonzero(mask == 0)[0]
    o = int(obs[len(obs) // 2])
    prev_action = int(np.nonzero(mask[:o] == 1)[0][-1])
    a = rew.copy(); a[o] = 0.7
    b = rew.copy(); b[prev_action] = 0.7
    cu = np.array([0, 120])
    ra = advantage(vals, a, mask, cu, 0.95, 0.8)
    rb = advantage(vals, b, mask, cu, 0.95, 0.8)
    assert np.allclose(ra[0], rb[0], atol=1e-13) and np.allclose(ra[1], rb[1], atol=1e-13)
    # a reward before the first action is dropped
    mask2 = mask.copy(); mask2[:3] = 0
    c = rew.copy(); c[0] = 5.0
    rc = advantage(vals, c, mask2, cu, 0.95, 0.8)
    rd = advantage(vals, rew, mask2, cu, 0.95, 0.8)
    assert np.array_equal(rc[0], rd[0]) and np.array_equal(rc[1], rd[1])


def test_constant_values_length_adaptive_closed_form():
    # V_t = v, one terminal reward R, gamma = 1: A_k = lambda_b^{n-1-k} (R - v)
    n_tok = 200
    rng = np.random.default_rng(14)
    mask = (rng.random(n_tok) > 0.3).astype(np.uint8); mask[-1] = 1
    vals = np.full(n_tok, 0.25, np.float32)
    rew = np.zeros(n_tok, np.float32); rew[-1] = 1.0
    adv, _, _ = advantage(vals, rew, mask, np.array([0, n_tok]), 1.0, 1.0, alpha=1.5)
    lam_b = 1.0 - 1.0 / (1.5 * n_tok)
    idx = np.nonzero(mask)[0]
    n = idx.size
    expect = np.array([lam_b ** (n - 1 - k) * 0.75 for k in range(n)])
    assert np.allclose(adv[idx], expect, rtol=1e-12, atol=1e-14)


def test_lambda_rule():
    assert trajectory_lambda(100, 50, 0.9, 0.0) == 0.9
    assert trajectory_lambda(100, 50, 0.9, 1.5) == pytest.approx(1 - 1 / 150)
    assert trajectory_lambda(100, 50, 0.9, 1.5, "actions") == pytest.approx(1 - 1 / 75)
    assert trajectory_lambda(1, 1, 0.9, 0.5) == 0.0       # 1 - 1/(0.5) < 0 clamps to 0


def test_returns_are_lambda_one_advantage_plus_value():
    b = generate(CONFIGS["c3"], with_head=False)
    adv1, ret, _ = advantage(b.values, b.rewards, b.mask, b.cu_seqlens, 0.99, 1.0)
    m = b.mask == 1
    assert np.allclose(ret[m], adv1[m] + b.values[m], atol=1e-9)


def test_trajectory_permutation_invariance():
    b = generate(CONFIGS["c0"], with_head=False)
    cu = b.cu_seqlens
    adv, ret, N = advantage(b.values, b.rewards, b.mask, cu, 0.99, 0.9, alpha=1.5)
    order = [2, 0, 3, 1]
    segs = [np.arange(cu[i], cu[i + 1]) for i in order]
    perm = np.concatenate(segs)
    cu2 = np.concatenate([[0], np.cumsum([s.size for s in segs])])
    adv2, ret2, N2 = advantage(b.values[perm], b.rewards[perm], b.mask[perm], cu2, 0.99, 0.9, alpha=1.5)
    assert N == N2
    assert np.array_equal(adv2, adv[perm]) and np.array_equal(ret2, ret[perm])


def test_empty_and_all_observation_trajectories():
    vals = np.ones(6, np.float32)
    rew = np.ones(6, np.float32)
    mask = np.zeros(6, np.uint8)
    adv, ret, N = advantage(vals, rew, mask, np.array([0, 0, 3, 6]), 1.0, 1.0)
    assert N == 0 and (adv == 0).all() and (ret == 0).all()
