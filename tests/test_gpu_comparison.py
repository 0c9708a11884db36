"""GPU parity of the comparison objectives (clipped surrogate of Sec. 2, clip-higher,
decoupled three-policy form of Sec. 3.1) and of the explained variance (Sec. 4.4)
against the fp64 oracle, through the C ABI.

Both sides read the same float32 inputs and compute in float64, so the bars are
tight: flags and counts bit-exact (the drift noise keeps every log-ratio at least
4e-3 from a clip edge, except in the edge tests, which place ratios within 1e-6
and check that the flags still agree), loss |d| <= 1e-9 (1/N) sum |terms|,
g within one float32 rounding (1e-6 relative), EV and the running moments within
1e-10 relative (the two sides accumulate in different orders).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2607_07508_amd as sao
from synth import CONFIGS, comparison_logprobs, generate, small_config, with_overrides
from tests.gpu_common import say

pytestmark = pytest.mark.gpu


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _scan_inputs(cfg):
    b = generate(cfg, with_head=False)
    adv, ret, n = oracle.advantage(b.values, b.rewards, b.mask, b.cu_seqlens, cfg.gamma, cfg.lam, cfg.alpha)
    return b, adv.astype(np.float32), ret.astype(np.float32), n


def _term_scale(lp, lold, lb, adv, mask, N):
    w = np.ones(lp.size) if lb is None else np.exp(lold.astype(np.float64) - lb)
    r = np.exp(lp.astype(np.float64) - lold)
    m = (mask != 0) & np.isfinite(r * w)
    return float(np.sum(np.abs(w * np.maximum(r, 1.0) * adv)[m])) / max(N, 1)


def _check_ppo(got, ref, scale):
    loss, g, flags, counts = (x.cpu().numpy() for x in got)
    rl, rg, rf, rc = ref
    assert np.array_equal(flags, rf), int((flags != rf).sum())
    assert np.array_equal(counts, rc), (counts, rc)
    assert abs(loss[0] - rl) <= 1e-9 * scale + 1e-300, (loss[0], rl)
    assert np.all(np.abs(g - rg) <= 1e-6 * np.abs(rg)), float(np.max(np.abs(g - rg)))


PPO_CASES = [
    # name, config, eps_low, eps_high, decoupled, global N
    ("c0-sym", CONFIGS["c0"], 0.2, 0.2, False, False),
    ("mid-3001-clip-higher", small_config("p1", 81, B=5, T=3001, H=8, V=8, eps_low=0.2, eps_high=0.28),
     0.2, 0.28, False, True),
    ("mid-20000-decoupled", small_config("p2", 82, B=9, T=20000, H=8, V=8, eps_low=0.2, eps_high=0.28),
     0.2, 0.28, True, True),
    ("c2-sym", CONFIGS["c2"], 0.2, 0.2, False, True),
    ("c2-decoupled-paper-pair", with_overrides(CONFIGS["c2"], eps_low=0.3, eps_high=5.0), 0.3, 5.0, True, True),
    ("c3-clip-higher", with_overrides(CONFIGS["c3"], eps_high=0.28), 0.2, 0.28, False, True),
]


@pytest.mark.parametrize("name,cfg,eps_low,eps_high,decoupled,global_n", PPO_CASES, ids=[c[0] for c in PPO_CASES])
def test_ppo_matches_oracle(name, cfg, eps_low, eps_high, decoupled, global_n):
    say(f"ppo parity {name}")
    b, adv, _, N = _scan_inputs(cfg)
    lp, lold, lb = comparison_logprobs(cfg, b.T)
    lb = lb if decoupled else None
    got = sao.ppo_loss(_t(lp), _t(lold), _t(adv), _t(b.mask), eps_low, eps_high,
                       _t(np.array([N], np.int64)) if global_n else None, None if lb is None else _t(lb))
    torch.cuda.synchronize()
    ref = oracle.ppo_loss(lp, lold, adv, b.mask, eps_low, eps_high, N, logp_behav=lb)
    assert ref[3][1] > 0 and ref[3][2] + ref[3][3] > 0
    _check_ppo(got, ref, _term_scale(lp, lold, lb, adv, b.mask, N))


@pytest.mark.parametrize("eps_low,eps_high", [(0.2, 0.28), (0.3, 5.0), (0.8, 3.0)])
def test_ppo_clip_decisions_near_edges(eps_low, eps_high):
    """Ratios within 1e-6 of either clip edge (in log space) flag exactly as in float64."""
    rng = np.random.default_rng(91)
    n = 8192
    lold = rng.uniform(-6.0, -0.05, n).astype(np.float32)
    edges = np.array([np.log1p(-eps_low), np.log1p(eps_high)])
    d = edges[rng.integers(0, 2, n)] + rng.uniform(-1e-6, 1e-6, n)
    lp = (lold.astype(np.float64) + d).astype(np.float32)
    adv = rng.normal(0.0, 1.0, n).astype(np.float32)
    mask = np.ones(n, dtype=np.uint8)
    mask[::13] = 0
    got = sao.ppo_loss(_t(lp), _t(lold), _t(adv), _t(mask), eps_low, eps_high)
    torch.cuda.synchronize()
    ref = oracle.ppo_loss(lp, lold, adv, mask, eps_low, eps_high)
    assert ref[3][2] > 100 and ref[3][3] > 100 and ref[3][1] > 100
    _check_ppo(got, ref, _term_scale(lp, lold, None, adv, mask, int(mask.sum())))


def test_ppo_extremes_and_nonfinite():
    """No lower edge (eps_low >= 1), infinite and huge ratios of both advantage signs, a
    zero advantage, NaN ratios and NaN weights."""
    lp = np.array([-800.0, -0.5, 0.0, -3.0, np.inf, np.inf, -np.inf, -np.inf, np.nan, -1.0, 90.0, 90.0, -2.0, -2.0],
                  dtype=np.float32)
    lold = np.array([0.0, 0.0, 0.0, -3.0, 0.0, 0.0, 0.0, 0.0, 0.0, np.nan, -10.0, -10.0, -2.5, -2.5],
                    dtype=np.float32)
    lb = lold.copy()
    lb[12] = np.nan
    lb[13] = -40.0
    adv = np.array([-1.0, 0.5, 0.0, 1.0, 1.0, -1.0, 1.0, -1.0, 1.0, 1.0, 1.0, -1.0, 1.0, 2.0], dtype=np.float32)
    mask = np.ones(lp.size, dtype=np.uint8)
    for eps_low in (1.0, 1.5, 0.2):
        for behav in (None, lb):
            got = sao.ppo_loss(_t(lp), _t(lold), _t(adv), _t(mask), eps_low, 0.28, None,
                               None if behav is None else _t(behav))
            torch.cuda.synchronize()
            rl, rg, rf, rc = oracle.ppo_loss(lp, lold, adv, mask, eps_low, 0.28, logp_behav=behav)
            loss, g, flags, counts = (x.cpu().numpy() for x in got)
            assert np.array_equal(flags, rf), (eps_low, behav is None, flags, rf)
            assert np.array_equal(counts, rc)
            # r = +inf with A < 0 stays unclipped: the objective is -inf on both sides
            assert (loss[0] == rl) or math.isclose(loss[0], rl, rel_tol=1e-12), (loss[0], rl)
            # g is float32: a ratio of e^100 overflows it to inf, as float32(ref) does
            with np.errstate(over="ignore", invalid="ignore"):
                rg32 = rg.astype(np.float32)
                ok = (g == rg32) | (np.abs(g.astype(np.float64) - rg) <= 1e-6 * np.abs(rg))
            assert ok.all(), (g, rg)


def test_ppo_unaligned_and_chunked():
    """Arrays at odd offsets take the scalar path; chunked calls with the global N sum to
    the whole batch's loss and counts."""
    cfg = small_config("p3", 83, B=7, T=9001, H=8, V=8, eps_low=0.2, eps_high=0.28)
    b, adv, _, N = _scan_inputs(cfg)
    lp, lold, lb = comparison_logprobs(cfg, b.T)
    ref = oracle.ppo_loss(lp, lold, adv, b.mask, 0.2, 0.28, N, logp_behav=lb)

    def shifted(x):
        buf = torch.empty(x.size + 1, dtype=torch.from_numpy(x[:1]).dtype, device="cuda")
        buf[1:] = _t(x)
        return buf[1:]
    n_dev = _t(np.array([N], np.int64))
    got = sao.ppo_loss(shifted(lp), shifted(lold), shifted(adv), shifted(b.mask), 0.2, 0.28, n_dev, shifted(lb))
    torch.cuda.synchronize()
    scale = _term_scale(lp, lold, lb, adv, b.mask, N)
    _check_ppo(got, ref, scale)

    loss = torch.zeros(1, dtype=torch.float64, device="cuda")
    counts = torch.zeros(5, dtype=torch.int64, device="cuda")
    gs, fs = [], []
    for s, e in ((0, 1000), (1000, 1003), (1003, 6000), (6000, b.T)):
        _, g, f, _ = sao.ppo_loss(_t(lp[s:e]), _t(lold[s:e]), _t(adv[s:e]), _t(b.mask[s:e]), 0.2, 0.28, n_dev,
                                  _t(lb[s:e]), loss=loss, counts=counts)
        gs.append(g)
        fs.append(f)
    torch.cuda.synchronize()
    _check_ppo((loss, torch.cat(gs), torch.cat(fs), counts), ref, scale)


def test_ppo_empty_mask_and_zero_tokens():
    cfg = small_config("p4", 84, B=3, T=700, H=8, V=8)
    b, adv, _, _ = _scan_inputs(cfg)
    lp, lold, lb = comparison_logprobs(cfg, b.T)
    mask = np.zeros(b.T, np.uint8)
    loss, g, flags, counts = sao.ppo_loss(_t(lp), _t(lold), _t(adv), _t(mask), 0.2, 0.2, None, _t(lb))
    torch.cuda.synchronize()
    assert loss.item() == 0.0 and (g.cpu().numpy() == 0).all() and (flags.cpu().numpy() == 0).all()
    assert counts.cpu().numpy().tolist() == [0, 0, 0, 0, 0]
    e = torch.empty(0, dtype=torch.float32, device="cuda")
    loss, g, flags, counts = sao.ppo_loss(e, e, e, torch.empty(0, dtype=torch.uint8, device="cuda"), 0.2, 0.2)
    assert loss.item() == 0.0 and g.numel() == 0 and counts.sum().item() == 0


# --------------------------------------------------------------------------- #
# Explained variance.
# --------------------------------------------------------------------------- #
def _ev_ref_moments(values, ret, mask):
    m = mask != 0
    R = ret.astype(np.float64)[m]
    d = R - values.astype(np.float64)[m]
    if R.size == 0:
        return np.zeros(5)
    return np.array([R.size, R.mean(), np.sum((R - R.mean()) ** 2), d.mean(), np.sum((d - d.mean()) ** 2)])


def _check_ev(ev, moments, values, ret, mask):
    want = oracle.explained_variance(values, ret, mask)
    got = ev.item()
    if math.isnan(want):
        assert math.isnan(got)
    else:
        assert got == pytest.approx(want, rel=1e-10, abs=1e-12)
    mom = moments.cpu().numpy()
    ref = _ev_ref_moments(values, ret, mask)
    assert mom[0] == ref[0]
    assert np.allclose(mom, ref, rtol=1e-10, atol=1e-12 * max(1.0, float(np.abs(ref).max()))), (mom, ref)


EV_CASES = [("c0", CONFIGS["c0"]), ("mid-3001", small_config("e1", 85, B=5, T=3001, H=8, V=8)),
            ("c2", CONFIGS["c2"]), ("c3", CONFIGS["c3"]), ("c4", CONFIGS["c4"])]


@pytest.mark.parametrize("name,cfg", EV_CASES, ids=[c[0] for c in EV_CASES])
def test_ev_matches_oracle(name, cfg):
    say(f"explained variance parity {name}")
    b, _, ret, _ = _scan_inputs(cfg)
    ev, moments = sao.explained_variance(_t(b.values), _t(ret), _t(b.mask))
    torch.cuda.synchronize()
    _check_ev(ev, moments, b.values, ret, b.mask)


def test_ev_chunked_and_unaligned():
    cfg = small_config("e2", 86, B=9, T=20011, H=8, V=8)
    b, _, ret, _ = _scan_inputs(cfg)
    moments = torch.zeros(5, dtype=torch.float64, device="cuda")
    for s, e in ((0, 1), (1, 5000), (5000, 5003), (5003, b.T)):
        ev, moments = sao.explained_variance(_t(b.values[s:e]), _t(ret[s:e]), _t(b.mask[s:e]), moments)
    torch.cuda.synchronize()
    _check_ev(ev, moments, b.values, ret, b.mask)

    def shifted(x):
        buf = torch.empty(x.size + 1, dtype=torch.from_numpy(x[:1]).dtype, device="cuda")
        buf[1:] = _t(x)
        return buf[1:]
    ev, moments = sao.explained_variance(shifted(b.values), shifted(ret), shifted(b.mask))
    torch.cuda.synchronize()
    _check_ev(ev, moments, b.values, ret, b.mask)


def test_ev_degenerate_cases():
    rng = np.random.default_rng(87)
    T = 5000
    values = rng.normal(0.5, 0.2, T).astype(np.float32)
    ret = rng.normal(0.5, 0.5, T).astype(np.float32)
    mask = (rng.random(T) < 0.6).astype(np.uint8)
    # no loss-mask token: NaN, moments stay zero
    ev, mom = sao.explained_variance(_t(values), _t(ret), _t(np.zeros(T, np.uint8)))
    torch.cuda.synchronize()
    assert math.isnan(ev.item()) and (mom.cpu().numpy() == 0).all()
    # constant returns: Var(R) is exactly 0 on both sides
    const = np.full(T, 0.7, np.float32)
    ev, mom = sao.explained_variance(_t(values), _t(const), _t(mask))
    torch.cuda.synchronize()
    assert math.isnan(ev.item()) and mom[2].item() == 0.0
    assert math.isnan(oracle.explained_variance(values, const, mask))
    # V = R: EV is exactly 1
    ev, _ = sao.explained_variance(_t(ret), _t(ret), _t(mask))
    torch.cuda.synchronize()
    assert ev.item() == 1.0 == oracle.explained_variance(ret, ret, mask)
