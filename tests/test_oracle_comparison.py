"""Pins of the oracle's comparison objectives: the clipped surrogate of Sec. 2 (with
clip-higher and the decoupled three-policy weight of Sec. 3.1) and the explained
variance of Sec. 4.4."""
import math

import numpy as np
import pytest
import torch

from oracle import explained_variance, ppo_loss


def _drifted(seed, T, sigma=0.3, frac_masked=0.2):
    rng = np.random.default_rng(seed)
    lp = -rng.gamma(2.0, 1.5, T)
    lold = lp + rng.normal(0.0, sigma, T)
    adv = rng.normal(0.0, 1.0, T)
    mask = (rng.random(T) >= frac_masked).astype(np.uint8)
    return lp, lold, adv, mask


def test_hand_worked_clipping_table():
    # eps = 0.2 on both sides; the four sign/side combinations of Sec. 3.1's description
    # of standard clipping, evaluated by hand:
    #   r=1.5, A=+1: clipped high, term 1.2     r=1.5, A=-1: unclipped, term -1.5
    #   r=0.5, A=+1: unclipped, term 0.5        r=0.5, A=-1: clipped low, term -0.8
    # loss = -(1.2 - 1.5 + 0.5 - 0.8) / 4 = 0.15; g = -r A / 4 on the unclipped pair.
    lold = np.zeros(4)
    lp = np.log([1.5, 1.5, 0.5, 0.5])
    adv = np.array([1.0, -1.0, 1.0, -1.0])
    loss, g, flags, counts = ppo_loss(lp, lold, adv, np.ones(4, np.uint8), 0.2, 0.2)
    assert flags.tolist() == [3, 1, 1, 2]
    assert counts.tolist() == [4, 2, 1, 1, 0]
    assert loss == pytest.approx(0.15, rel=1e-6)      # eps 0.2 is widened from float32
    assert g == pytest.approx([0.0, 1.5 / 4, -0.5 / 4, 0.0], rel=1e-12)


def test_clip_higher_moves_only_the_upper_edge():
    # eps_high = 0.28 > eps_low = 0.2: r = 1.25 with A > 0 is clipped at 0.2/0.2, kept at 0.2/0.28.
    lp = np.log([1.25, 0.75]).astype(np.float64)
    lold = np.zeros(2)
    adv = np.array([2.0, -1.0])
    sym = ppo_loss(lp, lold, adv, np.ones(2, np.uint8), 0.2, 0.2)
    hi = ppo_loss(lp, lold, adv, np.ones(2, np.uint8), 0.2, 0.28)
    assert sym[2].tolist() == [3, 2] and hi[2].tolist() == [1, 2]
    assert sym[0] == pytest.approx(-(1.2 * 2.0 - 0.8) / 2, rel=1e-6)
    assert hi[0] == pytest.approx(-(1.25 * 2.0 - 0.8) / 2, rel=1e-6)


def test_gradient_is_the_finite_difference_of_the_loss():
    lp, lold, adv, mask = _drifted(1, 64)
    eps_l, eps_h = 0.2, 0.28
    lo, hi = 1 - float(np.float32(eps_l)), 1 + float(np.float32(eps_h))
    r = np.exp(lp - lold)
    ok = (np.abs(np.log(r) - math.log(lo)) > 1e-3) & (np.abs(np.log(r) - math.log(hi)) > 1e-3)
    lp, lold, adv, mask = lp[ok], lold[ok], adv[ok], mask[ok]
    N = int(mask.sum())
    _, g, flags, _ = ppo_loss(lp, lold, adv, mask, eps_l, eps_h)
    assert (flags == 2).any() and (flags == 3).any() and (flags == 1).any()
    h = 1e-6
    for t in range(lp.size):
        up, dn = lp.copy(), lp.copy()
        up[t] += h
        dn[t] -= h
        fd = (ppo_loss(up, lold, adv, mask, eps_l, eps_h, N)[0] -
              ppo_loss(dn, lold, adv, mask, eps_l, eps_h, N)[0]) / (2 * h)
        assert fd == pytest.approx(g[t], rel=1e-6, abs=1e-9)


def test_gradient_matches_autograd_of_min_and_clamp():
    lp, lold, adv, mask = _drifted(2, 4096)
    behav = lold + np.random.default_rng(3).normal(0.0, 0.1, lold.size)
    eps_l, eps_h = 0.2, 0.28
    N = int(mask.sum())
    _, g, _, _ = ppo_loss(lp, lold, adv, mask, eps_l, eps_h, logp_behav=behav)
    x = torch.tensor(lp, dtype=torch.float64, requires_grad=True)
    r = torch.exp(x - torch.tensor(lold))
    w = torch.exp(torch.tensor(lold - behav))
    A = torch.tensor(adv)
    lo, hi = 1 - float(np.float32(eps_l)), 1 + float(np.float32(eps_h))
    obj = w * torch.minimum(r * A, torch.clamp(r, lo, hi) * A) * torch.tensor(mask, dtype=torch.float64)
    (-obj.sum() / N).backward()
    assert np.allclose(g, x.grad.numpy(), rtol=1e-12, atol=1e-18)


def test_wide_band_is_the_importance_weighted_surrogate():
    lp, lold, adv, mask = _drifted(4, 2048)
    loss, g, flags, counts = ppo_loss(lp, lold, adv, mask, 1.0, 1e30)
    m = mask == 1
    r = np.exp(lp - lold)
    assert counts.tolist() == [m.sum(), m.sum(), 0, 0, 0]
    assert loss == pytest.approx(-np.sum(r[m] * adv[m]) / m.sum(), rel=1e-12)
    assert np.allclose(g[m], -r[m] * adv[m] / m.sum(), rtol=1e-14)


def test_ratio_one_is_the_plain_advantage_mean():
    lp, _, adv, mask = _drifted(5, 1000)
    loss, g, flags, _ = ppo_loss(lp, lp, adv, mask, 0.2, 0.2)
    m = mask == 1
    assert (flags[m] == 1).all()
    assert loss == pytest.approx(-np.sum(adv[m]) / m.sum(), rel=1e-12, abs=1e-15)


def test_decoupled_weight_one_and_shift():
    lp, lold, adv, mask = _drifted(6, 3000)
    plain = ppo_loss(lp, lold, adv, mask, 0.2, 0.2)
    same = ppo_loss(lp, lold, adv, mask, 0.2, 0.2, logp_behav=lold)
    assert plain[0] == same[0] and np.array_equal(plain[1], same[1]) and np.array_equal(plain[2], same[2])
    c = 0.37        # pi_old / pi_behav scaled by e^c everywhere: loss and g scale, flags do not move
    shifted = ppo_loss(lp, lold, adv, mask, 0.2, 0.2, logp_behav=lold - c)
    assert np.array_equal(shifted[2], plain[2])
    assert shifted[0] == pytest.approx(math.exp(c) * plain[0], rel=1e-12)
    assert np.allclose(shifted[1], math.exp(c) * plain[1], rtol=1e-12)


def test_sign_of_advantage_picks_the_side():
    lp, lold, adv, mask = _drifted(7, 4000, sigma=0.5)
    pos = ppo_loss(lp, lold, np.abs(adv) + 1e-3, mask, 0.2, 0.2)[3]
    neg = ppo_loss(lp, lold, -np.abs(adv) - 1e-3, mask, 0.2, 0.2)[3]
    assert pos[2] == 0 and pos[3] > 0
    assert neg[3] == 0 and neg[2] > 0


def test_clip_counts_shrink_as_the_band_widens():
    lp, lold, adv, mask = _drifted(8, 5000, sigma=0.5)
    prev = None
    for eps in (0.1, 0.2, 0.3, 0.8):
        c = ppo_loss(lp, lold, adv, mask, eps, eps)[3]
        if prev is not None:
            assert c[2] <= prev[2] and c[3] <= prev[3]
        prev = c


def test_pessimistic_bound():
    # min(r A, clip(r) A) <= r A per token, so -N loss <= sum w r A.
    lp, lold, adv, mask = _drifted(9, 5000, sigma=0.5)
    behav = lold + 0.05
    loss, _, _, _ = ppo_loss(lp, lold, adv, mask, 0.2, 0.28, logp_behav=behav)
    m = mask == 1
    w = np.exp(lold - behav)
    assert -loss * m.sum() <= np.sum((w * np.exp(lp - lold) * adv)[m]) + 1e-9


def test_nan_ratio_is_flagged_and_adds_nothing():
    lp = np.array([np.nan, -1.0, -2.0])
    lold = np.array([-1.0, -1.0, np.nan])
    loss, g, flags, counts = ppo_loss(lp, lold, np.ones(3), np.ones(3, np.uint8), 0.2, 0.2)
    assert flags.tolist() == [4, 1, 4] and counts.tolist() == [3, 1, 0, 0, 2]
    assert loss == pytest.approx(-1.0 / 3) and g.tolist() == pytest.approx([0.0, -1.0 / 3, 0.0])


# --------------------------------------------------------------------------- #
# Explained variance (Sec. 4.4).
# --------------------------------------------------------------------------- #
def test_ev_matches_scikit_learn():
    from sklearn.metrics import explained_variance_score
    rng = np.random.default_rng(10)
    R = rng.normal(0.5, 1.0, 5000)
    V = R + rng.normal(0.0, 0.6, 5000)
    mask = (rng.random(5000) < 0.7).astype(np.uint8)
    m = mask == 1
    assert explained_variance(V, R, mask) == pytest.approx(explained_variance_score(R[m], V[m]), rel=1e-12)


@pytest.mark.parametrize("case,expect", [("exact", 1.0), ("offset", 1.0), ("const", 0.0),
                                         ("half", 0.75), ("double", 0.0), ("zero", 0.0)])
def test_ev_closed_forms(case, expect):
    R = np.random.default_rng(11).normal(1.0, 2.0, 999)
    V = {"exact": R, "offset": R + 3.0, "const": np.full_like(R, 7.0), "half": R / 2, "double": 2 * R,
         "zero": np.zeros_like(R)}[case]
    assert explained_variance(V, R, np.ones(R.size, np.uint8)) == pytest.approx(expect, abs=1e-12)


def test_ev_ignores_masked_tokens_and_degenerates_to_nan():
    rng = np.random.default_rng(12)
    R, V = rng.normal(size=100), rng.normal(size=100)
    mask = (np.arange(100) % 3 != 0).astype(np.uint8)
    V2 = V.copy()
    V2[mask == 0] = 1e6
    assert explained_variance(V, R, mask) == explained_variance(V2, R, mask)
    assert math.isnan(explained_variance(V, R, np.zeros(100, np.uint8)))
    assert math.isnan(explained_variance(V, np.full(100, 0.25), np.ones(100, np.uint8)))


def test_equality_at_an_edge_is_not_clipped():
    # Sec. 3.1 states standard clipping with strict inequalities: r = 1 + eps_high with A > 0,
    # and r = 1 - eps_low with A < 0, keep their gradient (both products are equal there).
    lp = np.log([2.0, 0.5])
    assert np.exp(lp).tolist() == [2.0, 0.5]
    loss, g, flags, _ = ppo_loss(lp, np.zeros(2), np.array([1.0, -1.0]), np.ones(2, np.uint8), 0.5, 1.0)
    assert flags.tolist() == [1, 1]
    assert g.tolist() == [-1.0, 0.25] and loss == pytest.approx(-(2.0 - 0.5) / 2, rel=1e-15)
