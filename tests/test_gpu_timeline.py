"""The per-workgroup timeline hook of the head kernels (a measurement hook, not
part of the pass): with it on, each of the four MFMA kernels writes one record
per tile it computes, its clock readings in order, and the pass's outputs stay
bit-identical to a run without it."""
import numpy as np
import pytest
import torch

import paper_2607_07508_amd as sao
from paper_2607_07508_amd import binding as B
from tests.gpu_common import say

pytestmark = pytest.mark.gpu

T, H, V = 3000, 512, 5000  # one backward vocabulary block of 5,120 rows; a ragged vocabulary tile


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    sao.lib()


@pytest.fixture(scope="module")
def inputs():
    gen = torch.Generator().manual_seed(71)
    hidden = (torch.randn(T, H, generator=gen) * 0.5).to(torch.bfloat16).cuda()
    w = (torch.randn(V, H, generator=gen) * 0.05).to(torch.bfloat16).cuda()
    target = torch.randint(0, V, (T,), generator=gen, dtype=torch.int32).cuda()
    g = torch.randn(T, generator=gen) * 1e-3
    g[torch.rand(T, generator=gen) < 0.4] = 0.0
    return hidden, w, target, g.cuda()


def _pass(hidden, w, target, g):
    logp, lse = sao.token_logprob(hidden, w, target)
    dh, dw = sao.loss_backward(hidden, w, target, lse, g)
    torch.cuda.synchronize()
    return logp, lse, dh, dw


def _tiles(m, n):
    return {(a, b) for a in range(-(-m // 256)) for b in range(-(-n // 256))}


@pytest.mark.parametrize("kernel", ["forward", "dz", "dH", "dW"])
def test_timeline_records_and_unchanged_outputs(inputs, kernel):
    hidden, w, target, g = inputs
    t_grad = int((g != 0).sum())
    kid, expect = {
        "forward": (B.KERNEL_HEAD_FORWARD, _tiles(V, T)),   # up to 8192 tokens one launch takes every tile
        "dz": (B.KERNEL_BACKWARD_DZ, _tiles(V, t_grad)),   # ditto, of the one vocabulary block
        "dH": (B.KERNEL_BACKWARD_DH, _tiles(t_grad, H)),
        "dW": (B.KERNEL_BACKWARD_DW, _tiles(V, H)),
    }[kernel]
    say(f"timeline hook on {kernel}: T={T} H={H} V={V} T_grad={t_grad}")
    ref = _pass(hidden, w, target, g)
    rec = torch.zeros((1 << 14, 8), dtype=torch.int64, device="cuda")
    try:
        B.clock_samples(rec, kid)
        got = _pass(hidden, w, target, g)
    finally:
        B.clock_samples(None)
    for a, b in zip(ref, got):
        assert torch.equal(a, b)
    r = rec.cpu().numpy()
    live = r[r[:, 2] > r[:, 1]]
    ran = live[live[:, 7] >= 0]
    tiles = [(int(x) >> 32, int(x) & 0xFFFFFFFF) for x in ran[:, 7]]
    # every tile once, or (dH with its K cut into pieces) every tile the same number of times
    counts = {t: tiles.count(t) for t in set(tiles)}
    assert set(counts) == expect
    assert len(set(counts.values())) == 1
    if kernel != "dH":
        assert set(counts.values()) == {1}
    # start <= after the prologue <= after the K loop <= end (shader clock), start < end (wall clock)
    assert (ran[:, 3] <= ran[:, 4]).all() and (ran[:, 4] <= ran[:, 5]).all() and (ran[:, 5] <= ran[:, 6]).all()
    assert (ran[:, 1] < ran[:, 2]).all()
    # after the hook is switched off, nothing records
    rec.zero_()
    _pass(hidden, w, target, g)
    assert int(rec.abs().sum()) == 0
