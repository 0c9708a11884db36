"""Host-side argument checks of the Python binding (no GPU needed).

The binding marshals raw pointers, so it rejects tensors of the wrong dtype,
layout, device or length before any library call: such a tensor would make a
kernel read past its end or misread its elements.
"""
import pytest
import torch

import paper_2607_07508_amd as sao


def _adv_args(T=64, B=2):
    values = torch.zeros(T, dtype=torch.float32)
    rewards = torch.zeros(T, dtype=torch.float32)
    mask = torch.ones(T, dtype=torch.uint8)
    cu = torch.tensor([0, T // 2, T], dtype=torch.int32)
    return values, rewards, mask, cu


@pytest.mark.parametrize("which,bad,err", [
    ("mask", torch.ones(64, dtype=torch.int32), TypeError),           # wrong dtype
    ("rewards", torch.zeros(63, dtype=torch.float32), ValueError),      # one element short
    ("rewards", torch.zeros(128, dtype=torch.float32)[::2], ValueError),  # strided view
    ("cu", torch.tensor([0, 32, 64], dtype=torch.int64), TypeError),   # int64 boundaries
])
def test_advantage_rejects_bad_arrays(which, bad, err):
    values, rewards, mask, cu = _adv_args()
    args = dict(values=values, rewards=rewards, mask=mask, cu=cu)
    args[which] = bad
    with pytest.raises(err):
        sao.advantage(args["values"], args["rewards"], args["mask"], args["cu"])


def test_clipped_loss_rejects_bad_arrays():
    T = 32
    lp = torch.zeros(T, dtype=torch.float32)
    mask = torch.ones(T, dtype=torch.uint8)
    with pytest.raises(TypeError):
        sao.clipped_loss(lp, torch.zeros(T, dtype=torch.float64), lp, mask, 0.2, 0.2)
    with pytest.raises(ValueError):
        sao.clipped_loss(lp, lp, torch.zeros(T - 1, dtype=torch.float32), mask, 0.2, 0.2)
    with pytest.raises(TypeError):
        sao.clipped_loss(lp, lp, lp, mask, 0.2, 0.2, n_tokens=torch.zeros(1, dtype=torch.int32))


def test_head_calls_reject_host_tensors_and_mismatched_shapes():
    h = torch.zeros(8, 16, dtype=torch.float32)
    w = torch.zeros(10, 16, dtype=torch.float32)
    tgt = torch.zeros(8, dtype=torch.int32)
    with pytest.raises(ValueError):       # host memory is not device memory
        sao.token_logprob(h, w, tgt)
    with pytest.raises(TypeError):
        sao.token_logprob(h, w.to(torch.bfloat16), tgt)
    with pytest.raises(ValueError):       # H differs
        sao.loss_backward(h, torch.zeros(10, 8), tgt, torch.zeros(8), torch.zeros(8))


def test_comparison_and_estimator_calls_reject_bad_arrays():
    T = 32
    lp = torch.zeros(T, dtype=torch.float32)
    mask = torch.ones(T, dtype=torch.uint8)
    with pytest.raises(TypeError):        # the decoupled weight's log-probs must be float32
        sao.ppo_loss(lp, lp, lp, mask, 0.2, 0.28, logp_behav=torch.zeros(T, dtype=torch.float64))
    with pytest.raises(ValueError):
        sao.ppo_loss(lp, lp, torch.zeros(T - 1), mask, 0.2, 0.28)
    with pytest.raises(TypeError):
        sao.explained_variance(lp, lp, mask, moments=torch.zeros(5, dtype=torch.float32))
    with pytest.raises(ValueError):
        sao.explained_variance(lp, lp, mask, moments=torch.zeros(4, dtype=torch.float64))
    values, rewards, mask, cu = _adv_args()
    with pytest.raises(ValueError):       # only "average" and "last"
        sao.step_advantage(values, rewards, mask, cu, step_value="median")
    with pytest.raises(TypeError):
        sao.step_advantage(values, rewards, mask.to(torch.int32), cu)
    with pytest.raises(TypeError):
        sao.group_advantage(rewards.double(), mask, cu, 2, 1e-6)
    history, seen = torch.zeros(3, 8, dtype=torch.float64), torch.zeros(3, dtype=torch.int64)
    with pytest.raises(ValueError):       # history is [n_keys, window]
        sao.running_mean_advantage(rewards, mask, cu, history.flatten(), seen)
    with pytest.raises(ValueError):
        sao.running_mean_advantage(rewards, mask, cu, history, seen[:2])
    with pytest.raises(TypeError):
        sao.running_mean_advantage(rewards, mask, cu, history, seen, keys=torch.zeros(2, dtype=torch.int64))
