"""Property checks of the oracle on many random inputs (hypothesis, fixed profile): facts of
the mathematics that a dropped term, a wrong sign or a swapped edge would break."""
import math

import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import explained_variance, ppo_loss, step_advantage

SETTINGS = settings(max_examples=60, deadline=None, derandomize=True)


@SETTINGS
@given(st.integers(1, 40), st.integers(0, 2**31 - 1), st.sampled_from([(0.2, 0.2), (0.2, 0.28), (0.3, 5.0)]))
def test_clipped_surrogate_is_continuous_in_logp(n, seed, eps):
    # min(r A, clip(r) A) is continuous in r, so nudging every log-prob by 1e-7 moves the
    # loss by at most about sum |w r A| 1e-7 / N, across clip edges included.
    rng = np.random.default_rng(seed)
    lold = rng.normal(-2.0, 1.0, n)
    # place some ratios right at the clip edges
    d = rng.choice([math.log1p(eps[1]), math.log1p(-eps[0]), 0.0], n) + rng.normal(0, 1e-8, n)
    lp = lold + d
    adv = rng.normal(0.0, 1.0, n)
    mask = np.ones(n, np.uint8)
    h = 1e-7
    a = ppo_loss(lp, lold, adv, mask, eps[0], eps[1])[0]
    b = ppo_loss(lp + h, lold, adv, mask, eps[0], eps[1])[0]
    bound = 2.0 * np.sum(np.abs(np.exp(lp + h - lold) * adv)) * h / n + 1e-15
    assert abs(b - a) <= bound


@SETTINGS
@given(st.integers(3, 200), st.integers(0, 2**31 - 1), st.floats(-5.0, 5.0), st.floats(0.1, 10.0))
def test_explained_variance_is_affine_invariant(n, seed, shift, scale):
    rng = np.random.default_rng(seed)
    R = rng.normal(0.0, 1.0, n)
    V = R + rng.normal(0.0, 0.5, n)
    mask = (rng.random(n) < 0.8).astype(np.uint8)
    mask[:2] = 1
    a = explained_variance(V, R, mask)
    b = explained_variance(scale * V + shift, scale * R + shift, mask)
    assert (math.isnan(a) and math.isnan(b)) or abs(a - b) <= 1e-9 * max(1.0, abs(a))


@SETTINGS
@given(st.integers(2, 80), st.integers(0, 2**31 - 1), st.sampled_from(["average", "last"]))
def test_step_gae_telescopes_at_lambda_one(T, seed, form):
    # gamma = lambda = 1: every step's advantage is the rewards from its start to the end of
    # the trajectory minus its own step value.
    rng = np.random.default_rng(seed)
    mask = (rng.random(T) < 0.6).astype(np.uint8)
    values = rng.normal(0.0, 1.0, T)
    rewards = rng.normal(0.0, 1.0, T)
    cu = np.array([0, T], np.int32)
    adv, ret, last, _ = step_advantage(values, rewards, mask, cu, 1.0, 1.0, 0.0, form)
    t = 0
    while t < T:
        if mask[t] and (t == 0 or not mask[t - 1]):
            z = t
            while z < T and mask[z]:
                z += 1
            v = values[t:z].mean() if form == "average" else values[z - 1]
            assert abs(adv[t] - (rewards[t:].sum() - v)) <= 1e-9 * (1 + abs(adv[t]))
            assert abs(ret[t] - rewards[t:].sum()) <= 1e-9 * (1 + abs(ret[t]))
            t = z
        else:
            t += 1
