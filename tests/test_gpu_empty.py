"""An empty batch (T = 0) through every binding call: no library call is made (empty
tensors carry null pointers), outputs are empty, accumulators untouched, N = 0."""
import pytest
import torch

import paper_2607_07508_amd as sao

pytestmark = pytest.mark.gpu


def test_every_call_accepts_an_empty_batch():
    dev = torch.device("cuda")
    f32 = torch.empty(0, dtype=torch.float32, device=dev)
    u8 = torch.empty(0, dtype=torch.uint8, device=dev)
    i32 = torch.empty(0, dtype=torch.int32, device=dev)
    cu = torch.zeros(2, dtype=torch.int32, device=dev)            # one empty trajectory
    hid = torch.empty((0, 64), dtype=torch.bfloat16, device=dev)
    w = torch.zeros((100, 64), dtype=torch.bfloat16, device=dev)
    wv = torch.zeros(64, dtype=torch.bfloat16, device=dev)
    logp, lse = sao.token_logprob(hid, w, i32, u8)
    assert logp.numel() == 0 and lse.numel() == 0
    adv, ret, n = sao.advantage(f32, f32, u8, cu)
    assert adv.numel() == 0 and int(n.item()) == 0
    sadv, sret, last, sn = sao.step_advantage(f32, f32, u8, cu)
    assert sadv.numel() == 0 and int(sn.item()) == 0
    loss = torch.full((2,), 3.0, dtype=torch.float64, device=dev)
    counts = torch.full((5,), 7, dtype=torch.int64, device=dev)
    sao.clipped_loss(f32, f32, f32, u8, 0.2, 0.2, loss=loss, counts=counts)
    sao.ppo_loss(f32, f32, f32, u8, 0.2, 0.2, loss=loss[:1], counts=counts)
    assert loss.tolist() == [3.0, 3.0] and counts.tolist() == [7] * 5
    ev, mom = sao.explained_variance(f32, f32, u8)
    assert torch.isnan(ev).all() and (mom == 0).all()
    dh, dw = sao.loss_backward(hid, w, i32, f32, f32)
    assert dh.numel() == 0 and (dw == 0).all()
    v = sao.value_forward(hid, wv)
    lv, dhv, dwv = sao.value_loss(hid, wv, v, f32, u8)
    assert v.numel() == 0 and lv.item() == 0.0 and (dwv == 0).all()
    gadv, ga, gr, gn = sao.group_advantage(f32, u8, cu, 1, 1e-6)
    history, seen = sao.running_mean_state(1, 4, dev)
    radv, ra, rr, rn = sao.running_mean_advantage(f32, u8, cu, history, seen)
    assert gadv.numel() == 0 and radv.numel() == 0 and int(seen.item()) == 0
    torch.cuda.synchronize()
