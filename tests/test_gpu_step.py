"""GPU parity of the step-level GAE (App. A.1) against the fp64 oracle, through the C ABI.

Bars: `last` and N bit-exact; advantages and returns |d| <= 1e-6 max(1, |ref|)
(float64 inside on both sides, rounded to float32 by the kernel).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_07508_amd as sao
from synth import CONFIGS, generate, small_config
from tests.gpu_common import TOL_ADV, say

pytestmark = pytest.mark.gpu


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _check(got, ref):
    adv, ret, last, n = got
    r_adv, r_ret, r_last, r_n = ref
    torch.cuda.synchronize()
    a, g = adv.cpu().numpy().astype(np.float64), ret.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(a - r_adv) <= TOL_ADV * np.maximum(1.0, np.abs(r_adv))), float(np.max(np.abs(a - r_adv)))
    assert np.all(np.abs(g - r_ret) <= TOL_ADV * np.maximum(1.0, np.abs(r_ret))), float(np.max(np.abs(g - r_ret)))
    assert np.array_equal(last.cpu().numpy(), r_last)
    assert int(n.item()) == r_n


def _run(values, rewards, mask, cu, gamma, lam, alpha, form):
    got = sao.step_advantage(_t(values), _t(rewards), _t(mask), _t(cu), gamma, lam, alpha, form)
    ref = oracle.step_advantage(values, rewards, mask, cu, gamma, lam, alpha, form)
    _check(got, ref)
    return ref


CASES = [("c0", CONFIGS["c0"]), ("mid-3001", small_config("st1", 111, B=5, T=3001, H=8, V=8)),
         ("mid-20000", small_config("st2", 112, B=37, T=20000, H=8, V=8)),
         ("c2", CONFIGS["c2"]), ("c3", CONFIGS["c3"]), ("c4", CONFIGS["c4"])]


@pytest.mark.parametrize("form", ["average", "last"])
@pytest.mark.parametrize("name,cfg", CASES, ids=[c[0] for c in CASES])
def test_step_gae_matches_oracle(name, cfg, form):
    say(f"step GAE parity {name} {form}")
    b = generate(cfg, with_head=False)
    ref = _run(b.values, b.rewards, b.mask, b.cu_seqlens, 1.0, 1.0, 1.5, form)
    assert ref[2].sum() >= cfg.B // 2          # the workload has steps to number
    _run(b.values, b.rewards, b.mask, b.cu_seqlens, 0.99, 0.9, 0.0, form)


def test_many_one_token_steps():
    """50,000 one-token steps in one trajectory: every thread of the recurrence takes a
    long chunk of steps. With a fixed lambda this is also the token-level GAE."""
    T = 100_001
    rng = np.random.default_rng(113)
    values = rng.normal(0.5, 0.2, T).astype(np.float32)
    rewards = (rng.random(T) < 0.01).astype(np.float32)
    mask = np.zeros(T, np.uint8)
    mask[1::2] = 1
    cu = np.array([0, T], np.int32)
    ref = _run(values, rewards, mask, cu, 1.0, 0.95, 0.0, "average")
    tok_adv, tok_ret, _ = oracle.advantage(values, rewards, mask, cu, 1.0, 0.95, 0.0)
    assert np.allclose(ref[0], tok_adv, rtol=1e-12, atol=1e-12) and np.allclose(ref[1], tok_ret, rtol=1e-12)
    _run(values, rewards, mask, cu, 1.0, 1.0, 1.5, "last")


def test_edge_trajectories():
    """Empty and observation-only trajectories, runs touching both ends of a trajectory,
    and neighbouring trajectories whose runs meet at the boundary (two steps, not one)."""
    mask = np.array([1, 1, 1,   1, 0, 1,   0, 0,   1,   0, 1, 1, 0], np.uint8)
    cu = np.array([0, 3, 3, 6, 8, 9, 13], np.int32)
    rng = np.random.default_rng(114)
    values = rng.normal(0.0, 1.0, mask.size).astype(np.float32)
    rewards = rng.normal(0.0, 1.0, mask.size).astype(np.float32)
    for form in ("average", "last"):
        ref = _run(values, rewards, mask, cu, 1.0, 0.7, 1.5, form)
        assert ref[2].tolist() == [0, 0, 1, 1, 0, 1, 0, 0, 1, 0, 0, 1, 0]


def test_unaligned_arrays_and_status_word():
    b = generate(small_config("st3", 115, B=6, T=5000, H=8, V=8))

    def shifted(x):
        buf = torch.empty(x.size + 1, dtype=torch.from_numpy(x[:1]).dtype, device="cuda")
        buf[1:] = _t(x)
        return buf[1:]
    got = sao.step_advantage(shifted(b.values), shifted(b.rewards), shifted(b.mask), _t(b.cu_seqlens), 1.0, 0.9,
                             1.5, "average")
    _check(got, oracle.step_advantage(b.values, b.rewards, b.mask, b.cu_seqlens, 1.0, 0.9, 1.5, "average"))
    # malformed segments: NaN outputs, last = 0, the status bit, and N still counted
    bad_cu = b.cu_seqlens.copy()
    bad_cu[2], bad_cu[3] = bad_cu[3], bad_cu[2]
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    adv, ret, last, n = sao.step_advantage(_t(b.values), _t(b.rewards), _t(b.mask), _t(bad_cu), 1.0, 1.0, 1.5,
                                           "last", status=status)
    torch.cuda.synchronize()
    assert status.item() & 2
    assert torch.isnan(adv).all() and torch.isnan(ret).all() and (last == 0).all()
    assert int(n.item()) == int(b.mask.sum())
