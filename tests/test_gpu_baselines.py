"""GPU parity of the critic-free baselines (GRPO's group normalisation, Sec. 2; the
running-mean reward window, Sec. 4.3 and 4.5) against the fp64 oracle, through the C ABI.

Bars: per-trajectory rewards and advantages (float64) within 1e-12 relative (the sums
run in a different order), token advantages within one float32 rounding, N exact, the
running-mean history ring within 1e-12 and its counts exact, NaN exactly where the
oracle has NaN.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2607_07508_amd as sao
from synth import CONFIGS, generate, small_config

pytestmark = pytest.mark.gpu


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _close(got, want, rel=1e-12):
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.all(np.abs(got[~nan] - want[~nan]) <= rel * np.maximum(1.0, np.abs(want[~nan]))), \
        float(np.max(np.abs(got[~nan] - want[~nan])))


def _check_tokens(adv, ref_adv):
    a = adv.cpu().numpy().astype(np.float64)
    nan = np.isnan(ref_adv)
    assert np.array_equal(np.isnan(a), nan)
    assert np.all(np.abs(a[~nan] - ref_adv[~nan]) <= 1e-6 * np.maximum(1.0, np.abs(ref_adv[~nan])))


def _dense_rewards(b, seed):
    # every token carries a reward, so the trajectory sums are long float64 sums
    return np.random.default_rng(seed).normal(0.0, 0.1, b.T).astype(np.float32)


GRPO_CASES = [("c0-g4", CONFIGS["c0"], 4, 1e-6, False), ("c0-g2-eps0", CONFIGS["c0"], 2, 0.0, False),
              ("mid-g8-dense", small_config("gr1", 131, B=32, T=9000, H=8, V=8), 8, 1e-6, True),
              ("c2-g8", CONFIGS["c2"], 8, 1e-6, False), ("c2-g4-eps0", CONFIGS["c2"], 4, 0.0, False),
              ("c4-g8-dense", CONFIGS["c4"], 8, 1e-4, True)]


@pytest.mark.parametrize("name,cfg,G,eps,dense", GRPO_CASES, ids=[c[0] for c in GRPO_CASES])
def test_grpo_matches_oracle(name, cfg, G, eps, dense):
    b = generate(cfg, with_head=False)
    rewards = _dense_rewards(b, 132) if dense else b.rewards
    adv, ta, tr, n = sao.group_advantage(_t(rewards), _t(b.mask), _t(b.cu_seqlens), G, eps)
    torch.cuda.synchronize()
    r_adv, r_A, r_R, r_n = oracle.group_advantage(rewards, b.mask, b.cu_seqlens, G, eps)
    _close(tr.cpu().numpy(), r_R)
    _close(ta.cpu().numpy(), r_A)
    _check_tokens(adv, r_adv)
    assert int(n.item()) == r_n


def _ring(history, n_keys, window):
    """Host-side ring state (history [n_keys, window], seen [n_keys]) of past-reward lists."""
    ring = np.zeros((n_keys, window))
    seen = np.zeros(n_keys, np.int64)
    for k, past in history.items():
        seen[k] = len(past)
        for j in range(max(0, len(past) - window), len(past)):
            ring[k, j % window] = past[j]
    return ring, seen


def _run_running_mean(rewards, mask, cu, window, n_keys, hist_lists, keys, state=None):
    history, seen = state if state is not None else (_t(_ring(hist_lists, n_keys, window)[0]),
                                                    _t(_ring(hist_lists, n_keys, window)[1]))
    adv, ta, tr, n = sao.running_mean_advantage(_t(rewards), _t(mask), _t(cu), history, seen,
                                                None if keys is None else _t(keys.astype(np.int32)))
    torch.cuda.synchronize()
    r_adv, r_A, r_R, r_n, r_hist = oracle.running_mean_advantage(rewards, mask, cu, window, hist_lists, keys)
    _close(tr.cpu().numpy(), r_R)
    _close(ta.cpu().numpy(), r_A)
    _check_tokens(adv, r_adv)
    assert int(n.item()) == r_n
    want_ring, want_seen = _ring(r_hist, n_keys, window)
    assert np.array_equal(seen.cpu().numpy(), want_seen)
    _close(history.cpu().numpy(), want_ring)
    return (history, seen), r_hist


@pytest.mark.parametrize("window,n_keys,keyed", [(128, 1, False), (8, 16, True), (3, 5, True)])
def test_running_mean_matches_oracle_over_two_batches(window, n_keys, keyed):
    """A history longer than the window, a batch longer than the window, then a second
    batch continuing from the state the first one left."""
    rng = np.random.default_rng(133 + window)
    hist = {k: list(rng.random(rng.integers(0, 3 * window))) for k in range(n_keys)}
    state = None
    for batch in range(2):
        b = generate(small_config(f"rm{batch}", 134 + batch, B=200, T=30000, H=8, V=8))
        rewards = _dense_rewards(b, 135 + batch)
        keys = rng.integers(0, n_keys, b.cfg.B) if keyed else None
        state, hist = _run_running_mean(rewards, b.mask, b.cu_seqlens, window, n_keys, hist, keys, state)


def test_running_mean_key_out_of_range_and_malformed_segments():
    b = generate(small_config("rm3", 136, B=12, T=3000, H=8, V=8))
    rewards = _dense_rewards(b, 137)
    keys = np.arange(12, dtype=np.int32) % 3
    keys[5] = 7                                     # outside [0, 3)
    history, seen = sao.running_mean_state(3, 4, "cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    adv, ta, tr, n = sao.running_mean_advantage(_t(rewards), _t(b.mask), _t(b.cu_seqlens), history, seen,
                                                _t(keys), status=status)
    torch.cuda.synchronize()
    assert status.item() & sao.binding.STATUS_KEY_RANGE
    A = ta.cpu().numpy()
    assert math.isnan(A[5]) and not np.isnan(np.delete(A, 5)).any()
    s, e = b.cu_seqlens[5], b.cu_seqlens[6]
    m = b.mask[s:e] == 1
    assert torch.isnan(adv[s:e][torch.from_numpy(m).cuda()]).all()
    ok = keys != 7
    r_adv, r_A, _, _, r_hist = oracle.running_mean_advantage(rewards[np.repeat(ok, np.diff(b.cu_seqlens))],
                                                             b.mask[np.repeat(ok, np.diff(b.cu_seqlens))],
                                                             np.concatenate([[0], np.cumsum(np.diff(b.cu_seqlens)[ok])]),
                                                             4, None, keys[ok])
    _close(A[ok], r_A)
    assert seen.cpu().numpy().tolist() == [len(r_hist[k]) for k in range(3)]
    # malformed segments: NaN outputs, status bit, history untouched
    before = (history.clone(), seen.clone())
    bad = b.cu_seqlens.copy()
    bad[-1] += 1
    status.zero_()
    adv, ta, tr, n = sao.running_mean_advantage(_t(rewards), _t(b.mask), _t(bad), history, seen, _t(keys % 3),
                                                status=status)
    torch.cuda.synchronize()
    assert status.item() & sao.binding.STATUS_SEGMENTS
    assert torch.isnan(adv).all() and torch.isnan(ta).all()
    assert torch.equal(history, before[0]) and torch.equal(seen, before[1])
    assert int(n.item()) == int(b.mask.sum())
    adv, ta, tr, n = sao.group_advantage(_t(rewards), _t(b.mask), _t(bad), 4, 1e-6, status=status)
    torch.cuda.synchronize()
    assert torch.isnan(adv).all() and torch.isnan(ta).all() and torch.isnan(tr).all()


def test_loss_mask_count_with_many_trajectories():
    """Thousands of workgroups add their loss-mask counts into the shared count slots:
    every advantage entry point still reports N exactly, and the advantages match."""
    b = generate(small_config("many", 138, B=5000, T=120000, H=8, V=8))
    N = int(b.mask.sum())
    args = (_t(b.values), _t(b.rewards), _t(b.mask), _t(b.cu_seqlens))
    adv, ret, n = sao.advantage(*args, 1.0, 0.9, 1.5)
    sadv, sret, last, sn = sao.step_advantage(*args, 1.0, 0.9, 1.5, "average")
    gadv, ga, gr, gn = sao.group_advantage(_t(b.rewards), _t(b.mask), _t(b.cu_seqlens), 8, 1e-6)
    history, seen = sao.running_mean_state(1, 128, "cuda")
    radv, ra, rr, rn = sao.running_mean_advantage(_t(b.rewards), _t(b.mask), _t(b.cu_seqlens), history, seen)
    torch.cuda.synchronize()
    assert [int(x.item()) for x in (n, sn, gn, rn)] == [N] * 4
    r_adv, r_ret, r_n = oracle.advantage(b.values, b.rewards, b.mask, b.cu_seqlens, 1.0, 0.9, 1.5)
    _check_tokens(adv, r_adv)
    s_adv, s_ret, s_last, _ = oracle.step_advantage(b.values, b.rewards, b.mask, b.cu_seqlens, 1.0, 0.9, 1.5,
                                                    "average")
    _check_tokens(sadv, s_adv)
    assert np.array_equal(last.cpu().numpy(), s_last)
    _close(ga.cpu().numpy(), oracle.group_advantage(b.rewards, b.mask, b.cu_seqlens, 8, 1e-6)[1])
    _close(ra.cpu().numpy(), oracle.running_mean_advantage(b.rewards, b.mask, b.cu_seqlens, 128)[1])
