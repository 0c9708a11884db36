"""Pins of the oracle's log-prob (Eq. 1-2): invariants, closed forms, library routines."""
import math

import numpy as np
import pytest
import scipy.special
import torch

from oracle import token_logprob, token_logprob_loop
from synth import CONFIGS, generate


def _rand(seed, T, H, V, scale=1.0):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((T, H)) * scale
    w = rng.standard_normal((V, H)) * scale
    y = rng.integers(0, V, size=T).astype(np.int32)
    return h, w, y


def test_softmax_sums_to_one():
    h, w, _ = _rand(1, 5, 8, 13)
    probs = np.zeros((5, 13))
    for v in range(13):
        lp, _ = token_logprob(h, w, np.full(5, v, np.int32))
        probs[:, v] = np.exp(lp)
    assert np.abs(probs.sum(axis=1) - 1.0).max() <= 1e-12


def test_logp_nonpositive_c0():
    b = generate(CONFIGS["c0"])
    lp, lse = token_logprob(b.hidden, b.w_head, b.target, b.mask)
    assert (lp[b.mask == 1] <= 0).all()
    assert (lp[b.mask == 0] == 0).all() and (lse[b.mask == 0] == 0).all()


@pytest.mark.parametrize("V", [1000, 151936])
def test_zero_weights_give_uniform(V):
    h = np.random.default_rng(2).standard_normal((3, 4))
    w = np.zeros((V, 4))
    lp, lse = token_logprob(h, w, np.array([0, V // 2, V - 1], np.int32))
    assert np.abs(lp + math.log(V)).max() <= 1e-12
    assert np.abs(lse - math.log(V)).max() <= 1e-12


def test_matches_scipy_logsumexp():
    h, w, y = _rand(3, 7, 6, 50, scale=1.5)
    lp, lse = token_logprob(h, w, y)
    z = h @ w.T
    ref = scipy.special.logsumexp(z, axis=1)
    assert np.allclose(lse, ref, rtol=1e-13, atol=0)
    assert np.allclose(lp, z[np.arange(7), y] - ref, rtol=1e-12, atol=1e-13)


def test_matches_torch_log_softmax():
    h, w, y = _rand(4, 9, 5, 8, scale=2.0)
    lp, _ = token_logprob(h, w, y)
    ref = torch.log_softmax(torch.tensor(h) @ torch.tensor(w).T, dim=1)
    ref = ref[torch.arange(9), torch.tensor(y, dtype=torch.long)].numpy()
    assert np.allclose(lp, ref, rtol=0, atol=1e-13)


@pytest.mark.parametrize("kappa", [0.0, 5.0, 30.0, 80.0])
def test_planted_peak_closed_form(kappa):
    # h = e_0 makes z_{t,v} = W[v, 0]; all logits 0 except the target at kappa.
    V = 1000
    w = np.zeros((V, 3))
    w[417, 0] = kappa
    h = np.array([[1.0, 0.0, 0.0]])
    lp, _ = token_logprob(h, w, np.array([417], np.int32))
    expect = kappa - math.log(math.exp(kappa) + (V - 1))
    assert abs(lp[0] - expect) <= 1e-12 * max(1.0, abs(expect))
    lp2, _ = token_logprob(h, w, np.array([3], np.int32))
    assert abs(lp2[0] - (0.0 - math.log(math.exp(kappa) + (V - 1)))) <= 1e-12 * (1 + kappa)


def test_vectorised_equals_loops_c0_subset():
    b = generate(CONFIGS["c0"])
    rows = np.nonzero(b.mask)[0][:6]
    m = np.zeros_like(b.mask)
    m[rows] = 1
    lp, lse = token_logprob(b.hidden, b.w_head[:200], np.minimum(b.target, 199), m)
    lp2, lse2 = token_logprob_loop(b.hidden, b.w_head[:200], np.minimum(b.target, 199), m)
    assert np.allclose(lp, lp2, rtol=1e-12, atol=1e-13)
    assert np.allclose(lse, lse2, rtol=1e-12, atol=1e-13)


def test_rows_subset_matches_full():
    h, w, y = _rand(5, 20, 4, 30)
    full, _ = token_logprob(h, w, y)
    sub, _ = token_logprob(h, w, y, rows=[3, 11, 19])
    assert np.array_equal(sub[[3, 11, 19]], full[[3, 11, 19]])
    assert (np.delete(sub, [3, 11, 19]) == 0).all()
