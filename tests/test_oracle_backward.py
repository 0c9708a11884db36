"""Pins of the oracle's backward through the log-softmax into hidden states and W_head."""
import numpy as np
import pytest
import torch

from oracle import (advantage, dis_loss, loss_backward, loss_backward_loop, surrogate_S,
                    token_logprob, value_forward, value_loss)
from synth import rollout_logprobs


def _tiny(seed, T=24, H=6, V=13, scale=0.7):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((T, H)) * scale
    w = rng.standard_normal((V, H)) * scale
    y = rng.integers(0, V, T).astype(np.int32)
    mask = (rng.random(T) > 0.25).astype(np.uint8)
    vals = rng.normal(0.5, 0.2, T)
    rew = np.zeros(T); rew[-1] = 1.0; mask[-1] = 1
    xi = rng.normal(0, 0.2, T)
    return h, w, y, mask, vals, rew, xi


def _grad_setup(seed):
    h, w, y, mask, vals, rew, xi = _tiny(seed)
    T = h.shape[0]
    lp, lse = token_logprob(h, w, y, mask)
    adv, _, N = advantage(vals, rew, mask, np.array([0, T // 2, T]), 0.95, 0.9)
    lro = rollout_logprobs(lp, xi).astype(np.float64)
    _, g, flags, _ = dis_loss(lp, lro, adv, mask, 0.2, 0.2)
    return h, w, y, mask, adv, lro, lse, g, flags, N


@pytest.mark.parametrize("seed", [0, 1])
def test_finite_differences_of_surrogate(seed):
    h, w, y, mask, adv, lro, lse, g, flags, N = _grad_setup(seed)
    assert (flags == 1).sum() >= 5
    dH, dW = loss_backward(h, w, y, lse, g)
    used = flags == 1
    eps = 1e-6

    def S(hh, ww):
        return surrogate_S(hh, ww, y, lro, adv, used, N)

    fd_h = np.zeros_like(h)
    for i in range(h.shape[0]):
        for k in range(h.shape[1]):
            hp, hm = h.copy(), h.copy()
            hp[i, k] += eps; hm[i, k] -= eps
            fd_h[i, k] = (S(hp, w) - S(hm, w)) / (2 * eps)
    fd_w = np.zeros_like(w)
    for v in range(w.shape[0]):
        for k in range(w.shape[1]):
            wp, wm = w.copy(), w.copy()
            wp[v, k] += eps; wm[v, k] -= eps
            fd_w[v, k] = (S(h, wp) - S(h, wm)) / (2 * eps)
    assert np.linalg.norm(dH - fd_h) <= 1e-6 * np.linalg.norm(fd_h)
    assert np.linalg.norm(dW - fd_w) <= 1e-6 * np.linalg.norm(fd_w)


def test_matches_torch_autograd():
    h, w, y, mask, adv, lro, lse, g, flags, N = _grad_setup(2)
    dH, dW = loss_backward(h, w, y, lse, g)
    th = torch.tensor(h, requires_grad=True)
    tw = torch.tensor(w, requires_grad=True)
    lp = torch.log_softmax(th @ tw.T, dim=1)[torch.arange(h.shape[0]), torch.tensor(y, dtype=torch.long)]
    used = torch.tensor(flags == 1)
    rho = torch.exp(lp - torch.tensor(lro)).detach()          # f(r) as a stop-gradient weight
    loss = -(torch.where(used, rho * torch.tensor(adv) * lp, torch.zeros(()))).sum() / N
    loss.backward()
    assert np.allclose(dH, th.grad.numpy(), rtol=1e-10, atol=1e-14)
    assert np.allclose(dW, tw.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_invariants_and_loops():
    h, w, y, mask, adv, lro, lse, g, flags, N = _grad_setup(3)
    dH, dW = loss_backward(h, w, y, lse, g)
    assert np.abs(dW.sum(axis=0)).max() <= 1e-13             # sum_v dz_{t,v} = 0
    assert (dH[g == 0] == 0).all()
    dH2, dW2 = loss_backward_loop(h, w, y, lse, g)
    assert np.allclose(dH, dH2, rtol=1e-12, atol=1e-15) and np.allclose(dW, dW2, rtol=1e-12, atol=1e-15)


def test_zero_weights_closed_form():
    h, w, y, mask, vals, rew, xi = _tiny(4)
    V = w.shape[0]
    w0 = np.zeros_like(w)
    g = np.random.default_rng(5).normal(0, 0.1, h.shape[0]) * mask
    lse = np.full(h.shape[0], np.log(V))
    dH, dW = loss_backward(h, w0, y, lse, g)
    assert (dH == 0).all()
    expect = np.zeros_like(w)
    for t in range(h.shape[0]):
        for v in range(V):
            expect[v] += g[t] * ((1.0 if v == y[t] else 0.0) - 1.0 / V) * h[t]
    assert np.allclose(dW, expect, rtol=1e-12, atol=1e-15)


def test_sampled_rows_match_full():
    h, w, y, mask, adv, lro, lse, g, flags, N = _grad_setup(6)
    dH, dW = loss_backward(h, w, y, lse, g)
    rows = np.nonzero(g)[0][:4]
    vrows = np.array([0, 5, int(y[rows[0]]), 12])
    sH, sW = loss_backward(h, w, y, lse, g, dh_rows=rows, dw_rows=vrows)
    assert np.allclose(sH[rows], dH[rows], rtol=1e-13, atol=1e-16)
    assert np.allclose(sW[vrows], dW[vrows], rtol=1e-13, atol=1e-16)
    assert (np.delete(sW, vrows, axis=0) == 0).all()


def test_value_loss_finite_differences_and_closed_form():
    h, _, _, mask, vals, rew, _ = _tiny(7, T=16, H=5)
    wv = np.random.default_rng(8).standard_normal(5) * 0.3
    v = value_forward(h, wv)
    assert np.allclose(v, h @ wv)
    G = np.random.default_rng(9).normal(0.5, 0.5, 16)
    L, dH, dw = value_loss(h, wv, v, G, mask)
    N = int(mask.sum())
    assert L == pytest.approx(float(((v - G) ** 2 * mask).sum() / N), rel=1e-12)
    eps = 1e-6

    def f(hh, ww):
        return value_loss(hh, ww, value_forward(hh, ww), G, mask)[0]

    fd_w = np.array([(f(h, wv + eps * e) - f(h, wv - eps * e)) / (2 * eps) for e in np.eye(5)])
    assert np.allclose(dw, fd_w, rtol=1e-6, atol=1e-9)
    i, k = 3, 2
    hp, hm = h.copy(), h.copy(); hp[i, k] += eps; hm[i, k] -= eps
    assert dH[i, k] == pytest.approx((f(hp, wv) - f(hm, wv)) / (2 * eps), rel=1e-6, abs=1e-9)
