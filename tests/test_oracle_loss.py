"""Pins of the oracle's DIS ratio, strict double-sided band and token mean (Eq. 1-3)."""
import math

import numpy as np
import pytest

from oracle import advantage, dis_loss, token_logprob
from synth import CONFIGS, generate, rollout_logprobs
from tests.golden.load import dis_example


def _c0():
    b = generate(CONFIGS["c0"])
    lp, _ = token_logprob(b.hidden, b.w_head, b.target, b.mask)
    adv, _, N = advantage(b.values, b.rewards, b.mask, b.cu_seqlens, 1.0, 1.0)
    return b, lp, adv, N


def test_golden_worked_example():
    ex = dis_example()
    loss, g, flags, counts = dis_loss(ex["logp"], ex["logp_rollout"], ex["adv"], ex["mask"],
                                      ex["eps_low"], ex["eps_high"])
    assert np.array_equal(flags, ex["flags"])
    assert np.array_equal(counts, ex["counts"])
    assert np.allclose(loss, ex["loss"], rtol=1e-12, atol=0)
    assert np.allclose(g, ex["g"], rtol=1e-12, atol=0)


def test_ratio_one_clips_nothing():
    b, lp, adv, N = _c0()
    lro = lp.astype(np.float32).astype(np.float64)
    loss, g, flags, counts = dis_loss(lro, lro, adv, b.mask, 0.2, 0.2)
    m = b.mask == 1
    assert (flags[m] == 1).all() and (flags[~m] == 0).all()
    assert counts.tolist() == [N, N, 0, 0, 0]
    assert loss[0] == pytest.approx(-np.sum(adv[m] * lro[m]) / N, rel=1e-12)
    assert loss[1] == pytest.approx(-np.sum(adv[m]) / N, rel=1e-12, abs=1e-15)


def test_flags_follow_the_drift_noise_alone():
    # log pi_rollout = log pi + xi, so the log-ratio is -xi up to float32 rounding of the
    # rollout log-prob; the guard band keeps -xi at least 4e-3 from both band edges.
    b, lp, adv, _ = _c0()
    lro = rollout_logprobs(lp, b.xi)
    _, _, flags, counts = dis_loss(lp, lro, adv, b.mask, b.cfg.eps_low, b.cfg.eps_high)
    m = b.mask == 1
    lo = np.log(1 - np.float64(np.float32(b.cfg.eps_low)))
    hi = np.log(1 + np.float64(np.float32(b.cfg.eps_high)))
    expect = np.where(-b.xi <= lo, 2, np.where(-b.xi >= hi, 3, 1))
    assert np.array_equal(flags[m], expect[m])
    assert counts[0] == counts[1:].sum()


def test_counts_partition_and_zero_gradient_off_band():
    b = generate(CONFIGS["c2"], with_head=False)
    lp = np.full(b.T, -11.9)
    adv, _, N = advantage(b.values, b.rewards, b.mask, b.cu_seqlens, 1.0, 1.0, alpha=1.5)
    lro = rollout_logprobs(lp, b.xi)
    loss, g, flags, counts = dis_loss(lp, lro, adv, b.mask, 0.2, 0.2)
    assert counts[0] == N == counts[1:].sum()
    assert (g[flags != 1] == 0).all()
    assert 0.25 < (counts[2] + counts[3]) / N < 0.4      # sigma = 0.2 drift: about 31% clipped


def test_linear_in_advantage():
    b, lp, adv, _ = _c0()
    lro = rollout_logprobs(lp, b.xi)
    l1, g1, f1, _ = dis_loss(lp, lro, adv, b.mask, 0.2, 0.2)
    l2, g2, f2, _ = dis_loss(lp, lro, -2.5 * adv, b.mask, 0.2, 0.2)
    assert np.array_equal(f1, f2)
    assert np.allclose(l2, -2.5 * l1, rtol=1e-12) and np.allclose(g2, -2.5 * g1, rtol=1e-12)


def test_band_edges_are_strict():
    lp = np.array([-1.0, -1.0], np.float32)
    one = dis_loss(lp, lp, np.ones(2), np.ones(2, np.uint8), 0.0, 0.0)
    assert one[2].tolist() == [2, 2]                       # rho = 1 = 1 - 0 is outside (1, 1)
    wide = dis_loss(lp, lp, np.ones(2), np.ones(2, np.uint8), 0.999, 1e30)
    assert wide[2].tolist() == [1, 1]


def test_nonfinite_and_extreme_ratios():
    lp = np.array([np.nan, 0.0, -np.inf, 50.0, -1.0], np.float64)
    lro = np.array([-1.0, np.inf, -1.0, -np.inf, np.nan])
    mask = np.ones(5, np.uint8)
    loss, g, flags, counts = dis_loss(lp, lro, np.ones(5), mask, 1.0, 0.2)
    # NaN; rho = 0 (lower edge 0 with eps_low = 1); rho = 0; rho = +inf; NaN
    assert flags.tolist() == [4, 2, 2, 3, 4]
    assert (g == 0).all() and (loss == 0).all()
    assert counts.tolist() == [5, 0, 2, 1, 2]


def test_lower_edge_past_one():
    """eps_low > 1 puts 1 - eps_low below 0. A ratio is never negative, so the lower
    edge is 0: every positive ratio below 1 + eps_high is used, and rho = 0 (log pi =
    -inf, or a log-ratio so low that exp underflows) is clipped low. The token's
    term is then left out rather than being 0 * -inf."""
    lp = np.array([-np.inf, -800.0, -0.5, -30.0], np.float64)
    lro = np.zeros(4)
    adv = np.array([1.0, -2.0, 3.0, 0.5])
    loss, g, flags, counts = dis_loss(lp, lro, adv, np.ones(4, np.uint8), 1.5, 0.2)
    assert flags.tolist() == [2, 2, 1, 1]
    assert counts.tolist() == [4, 2, 2, 0, 0]
    r2, r3 = math.exp(-0.5), math.exp(-30.0)
    # hand-worked: -(1/4)(r2 * 3 * -0.5 + r3 * 0.5 * -30)
    assert loss[0] == pytest.approx(-(r2 * 3 * -0.5 + r3 * 0.5 * -30.0) / 4, rel=1e-14)
    assert loss[1] == pytest.approx(-(r2 * 3 + r3 * 0.5) / 4, rel=1e-14)
    assert np.isfinite(loss).all() and g[0] == 0 and g[1] == 0
    # eps_low = 1 gives the same edge
    assert dis_loss(lp, lro, adv, np.ones(4, np.uint8), 1.0, 0.2)[2].tolist() == flags.tolist()


def test_global_token_count_and_empty():
    b, lp, adv, N = _c0()
    lro = rollout_logprobs(lp, b.xi)
    l1, g1, _, _ = dis_loss(lp, lro, adv, b.mask, 0.2, 0.2)
    l2, g2, _, c2 = dis_loss(lp, lro, adv, b.mask, 0.2, 0.2, n_tokens=4 * N)
    assert np.allclose(l2, l1 / 4, rtol=1e-12) and np.allclose(g2, g1 / 4, rtol=1e-12)
    assert c2[0] == N                                   # counts report this call's tokens
    z = dis_loss(lp, lro, adv, np.zeros_like(b.mask), 0.2, 0.2)
    assert (z[0] == 0).all() and (z[1] == 0).all() and z[3].tolist() == [0, 0, 0, 0, 0]


@pytest.mark.parametrize("eps_low,eps_high", [(0.3, 5.0), (0.8, 3.0), (0.2, 0.28)])
def test_paper_band_pairs(eps_low, eps_high):
    # The paper's two clip pairs (and the large-head workload's): log-ratios on a grid
    # across both edges, kept 1e-4 away from them, give flags that follow the ratio
    # alone; used tokens lie strictly inside (1 - eps_l, 1 + eps_h) and carry
    # g = -rho A / N, every other token exactly 0.
    lo = math.log(1.0 - float(np.float32(eps_low)))
    hi = math.log(1.0 + float(np.float32(eps_high)))
    d = np.linspace(lo - 1.5, hi + 1.0, 6001)
    d = d[(np.abs(d - lo) > 1e-4) & (np.abs(d - hi) > 1e-4)]
    lp = np.full(d.size, -2.0)
    lro = lp - d
    adv = np.linspace(-1.0, 1.0, d.size)
    mask = np.ones(d.size, dtype=np.uint8)
    _, g, flags, counts = dis_loss(lp, lro, adv, mask, eps_low, eps_high)
    expect = np.where(d < lo, 2, np.where(d > hi, 3, 1))
    assert np.array_equal(flags, expect)
    rho = np.exp(d)
    used = flags == 1
    assert ((rho[used] > 1.0 - eps_low - 1e-7) & (rho[used] < 1.0 + eps_high + 1e-7)).all()
    assert np.allclose(g[used], -rho[used] * adv[used] / d.size, rtol=1e-9, atol=0)
    assert (g[~used] == 0).all()
    assert counts.tolist() == [d.size, int(used.sum()), int((d < lo).sum()), int((d > hi).sum()), 0]
