"""Pins of the oracle's step-level GAE (App. A.1): one advantage per agentic step."""
import numpy as np
import pytest

from oracle import advantage, step_advantage, steps_of
from synth import CONFIGS, generate, small_config


def _example():
    # tokens:    0  1  2  3  4  5  6  7  8  9      (one trajectory)
    mask = np.array([0, 1, 1, 0, 0, 1, 1, 1, 0, 1], np.uint8)
    values = np.array([9, 1, 3, 9, 9, 2, 4, 6, 9, 5], np.float32)
    rewards = np.array([7, 0, 0, 1, 0, 0, 0, 0, 2, 3], np.float32)
    return values, rewards, mask, np.array([0, 10], np.int32)


def test_hand_worked_example():
    # Steps [1,3), [5,8), [9,10). Step rewards fold the following observations and drop
    # the reward before the first step: R = (0+0+1+0, 0+0+0+2, 3) = (1, 2, 3).
    # Average values (2, 4, 5); last-token values (3, 6, 5). gamma = 1, lambda = 0.5:
    #   average: delta = (1+4-2, 2+5-4, 3-5) = (3, 3, -2); A2 = -2, A1 = 3 - 1 = 2, A0 = 3 + 1 = 4
    #   last:    delta = (1+6-3, 2+5-6, 3-5) = (4, 1, -2); A2 = -2, A1 = 1 - 1 = 0, A0 = 4 + 0 = 4
    #   returns G = (6, 5, 3) in both forms.
    v, r, m, cu = _example()
    adv, ret, last, n = step_advantage(v, r, m, cu, 1.0, 0.5, 0.0, "average")
    assert adv.tolist() == [0, 4, 4, 0, 0, 2, 2, 2, 0, -2]
    assert ret.tolist() == [0, 6, 6, 0, 0, 5, 5, 5, 0, 3]
    assert last.tolist() == [0, 0, 1, 0, 0, 0, 0, 1, 0, 1] and n == 6
    adv, ret, _, _ = step_advantage(v, r, m, cu, 1.0, 0.5, 0.0, "last")
    assert adv.tolist() == [0, 4, 4, 0, 0, 0, 0, 0, 0, -2]
    assert ret.tolist() == [0, 6, 6, 0, 0, 5, 5, 5, 0, 3]


def test_length_adaptive_lambda_counts_steps():
    # Three steps and alpha = 1.5: lambda = 1 - 1/4.5 = 7/9 (not the 10-token length).
    v, r, m, cu = _example()
    adv, _, _, _ = step_advantage(v, r, m, cu, 1.0, 0.0, 1.5, "average")
    lam = 7.0 / 9.0
    a2 = -2.0
    a1 = 3.0 + lam * a2
    a0 = 3.0 + lam * a1
    assert adv[[1, 5, 9]] == pytest.approx([a0, a1, a2], rel=1e-15)


@pytest.mark.parametrize("mode", ["average", "last"])
def test_one_token_steps_are_the_token_level_gae(mode):
    # With every action token isolated by observations, each step is one token and
    # (for a fixed lambda) the step form is the token-level skip-observation GAE.
    b = generate(small_config("s1", 101, B=6, T=3000, H=8, V=8))
    mask = np.zeros(b.T, np.uint8)
    mask[1::2] = 1
    for s, e in zip(b.cu_seqlens[:-1], b.cu_seqlens[1:]):
        mask[s] = 0                     # keep runs inside trajectories
    a_tok, r_tok, n_tok = advantage(b.values, b.rewards, mask, b.cu_seqlens, 0.99, 0.9, 0.0)
    a_st, r_st, last, n_st = step_advantage(b.values, b.rewards, mask, b.cu_seqlens, 0.99, 0.9, 0.0, mode)
    assert n_tok == n_st and np.array_equal(last, mask)
    assert np.allclose(a_st, a_tok, rtol=1e-13, atol=1e-13)
    assert np.allclose(r_st, r_tok, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("mode", ["average", "last"])
def test_lambda_one_and_zero(mode):
    b = generate(CONFIGS["c0"])
    m = b.mask == 1
    a1, g1, last, _ = step_advantage(b.values, b.rewards, b.mask, b.cu_seqlens, 1.0, 1.0, 0.0, mode)
    a0, g0, _, _ = step_advantage(b.values, b.rewards, b.mask, b.cu_seqlens, 1.0, 0.0, 0.0, mode)
    assert np.array_equal(g1, g0)
    # lambda = gamma = 1 telescopes to A_i = G_i - V_i; lambda = 0 leaves the TD residual.
    for bi in range(b.cfg.B):
        steps = steps_of(b.mask, int(b.cu_seqlens[bi]), int(b.cu_seqlens[bi + 1]))
        V = [float(np.mean(b.values[a:z].astype(np.float64))) if mode == "average" else float(b.values[z - 1])
             for a, z in steps]
        for i, (a, z) in enumerate(steps):
            assert a1[a] == pytest.approx(g1[a] - V[i], abs=1e-12)
            v_next = V[i + 1] if i + 1 < len(steps) else 0.0
            r_i = g1[a] - (g1[steps[i + 1][0]] if i + 1 < len(steps) else 0.0)
            assert a0[a] == pytest.approx(r_i + v_next - V[i], abs=1e-12)
    assert (a1[~m] == 0).all() and (g1[~m] == 0).all()


def test_constant_step_values_make_both_forms_equal():
    b = generate(CONFIGS["c0"])
    vals = b.values.copy()
    for bi in range(b.cfg.B):
        for a, z in steps_of(b.mask, int(b.cu_seqlens[bi]), int(b.cu_seqlens[bi + 1])):
            vals[a:z] = vals[z - 1]
    x = step_advantage(vals, b.rewards, b.mask, b.cu_seqlens, 1.0, 0.95, 1.5, "average")
    y = step_advantage(vals, b.rewards, b.mask, b.cu_seqlens, 1.0, 0.95, 1.5, "last")
    assert np.allclose(x[0], y[0], rtol=1e-14, atol=1e-14) and np.array_equal(x[1], y[1])


def test_rewards_move_freely_inside_a_step_span():
    # A reward anywhere from a step's first token to the next step's first token is that
    # step's reward; moving it there changes nothing.
    v, r, m, cu = _example()
    r2 = r.copy()
    r2[3], r2[1] = 0.0, 1.0            # step 0's reward moved from an observation onto an action
    r2[8], r2[7] = 0.0, 2.0            # step 1's likewise
    for mode in ("average", "last"):
        x = step_advantage(v, r, m, cu, 0.97, 0.5, 0.0, mode)
        y = step_advantage(v, r2, m, cu, 0.97, 0.5, 0.0, mode)
        assert np.array_equal(x[0], y[0]) and np.array_equal(x[1], y[1])


def test_single_step_ignores_lambda_and_permutation_invariance():
    v = np.array([0.25, 0.5, 0.75, 0.0], np.float32)
    r = np.array([0.0, 0.0, 1.0, 0.5], np.float32)
    m = np.array([1, 1, 1, 0], np.uint8)
    cu = np.array([0, 4], np.int32)
    for alpha in (0.0, 1.5, 100.0):
        adv, ret, _, _ = step_advantage(v, r, m, cu, 1.0, 0.3, alpha, "average")
        assert adv[:3].tolist() == pytest.approx([1.5 - 0.5] * 3) and ret[:3].tolist() == [1.5] * 3
    # trajectories are independent: reversing their order permutes the outputs
    b = generate(CONFIGS["c0"])
    cu = b.cu_seqlens
    order = list(range(b.cfg.B))[::-1]
    idx = np.concatenate([np.arange(cu[i], cu[i + 1]) for i in order])
    lens = np.array([cu[i + 1] - cu[i] for i in order])
    cu2 = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    x = step_advantage(b.values, b.rewards, b.mask, cu, 1.0, 0.9, 1.5, "last")
    y = step_advantage(b.values[idx], b.rewards[idx], b.mask[idx], cu2, 1.0, 0.9, 1.5, "last")
    assert np.array_equal(x[0][idx], y[0]) and np.array_equal(x[1][idx], y[1]) and np.array_equal(x[2][idx], y[2])


def test_empty_and_observation_only_trajectories():
    v = np.ones(6, np.float32)
    r = np.ones(6, np.float32)
    m = np.array([0, 0, 0, 1, 1, 0], np.uint8)
    cu = np.array([0, 0, 3, 6], np.int32)          # empty, observation-only, one step
    adv, ret, last, n = step_advantage(v, r, m, cu, 1.0, 1.0, 1.5, "average")
    assert (adv[:3] == 0).all() and (ret[:3] == 0).all() and n == 2
    assert ret[3:5].tolist() == [3.0, 3.0] and last.tolist() == [0, 0, 0, 0, 1, 0]
