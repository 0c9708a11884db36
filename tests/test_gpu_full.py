"""Full-size parity in the launch configuration the benchmark times.

Log-probs and lse are compared on every loss-mask row against the oracle values
stored by tests/golden/make_full_logprobs.py; advantages, flags, counts, loss
and g on every token (the oracle scan and loss are cheap); dhidden and dW_head
on every element at c2 (the bench's workload), on sampled rows that the oracle
computes one by one at c3 and c4, plus exact zeros on every row with g = 0.
"""
import numpy as np
import pytest
import torch

import oracle
from synth import CONFIGS, generate, rollout_logprobs
from tests.gpu_common import (TOL_ADV, TOL_G, TOL_LOGP, check_grad, check_loss, check_value, gpu_pass,
                               say)
from tests.golden.make_full_logprobs import load as load_golden, path_for

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")


def _oracle_backward_every_row(b, ref_lse, g, w64, chunk=4096):
    """The oracle's dH and dW over every token and vocabulary row, computed over
    chunks of the rows with g != 0 (both are sums over tokens, so the chunks'
    dW add up to the whole), with a progress line per chunk."""
    live = np.nonzero(g)[0]
    dH = np.zeros((b.T, b.cfg.H), dtype=np.float64)
    dW = np.zeros((b.cfg.V, b.cfg.H), dtype=np.float64)
    for s in range(0, live.size, chunk):
        r = live[s:s + chunk]
        gc = np.zeros_like(g)
        gc[r] = g[r]
        dh_c, dw_c = oracle.loss_backward(b.hidden, None, b.target, ref_lse, gc, w64=w64)
        dH[r] = dh_c[r]
        dW += dw_c
        del dh_c, dw_c
        say(f"{b.cfg.name}: oracle backward rows {s + r.size} of {live.size}")
    return dH, dW


def _full(name, backward, n_rows=24, seed=0, every_row=False):
    cfg = CONFIGS[name]
    say(f"{name}: generating T={cfg.T} H={cfg.H} V={cfg.V}")
    b = generate(cfg)
    ref_lp, ref_lse = load_golden(name, b)
    say(f"{name}: GPU pass" + (f" in chunks of {cfg.chunk}" if cfg.chunk else ""))
    got = gpu_pass(b, ref_lp, cfg.gamma, cfg.lam, cfg.alpha, backward, chunk=cfg.chunk)
    m = b.mask == 1
    say(f"{name}: compare logp on {int(m.sum())} rows")
    assert np.abs(got["logp"][m] - ref_lp[m]).max() <= TOL_LOGP
    assert np.abs(got["lse"][m] - ref_lse[m]).max() <= TOL_LOGP
    assert (got["logp"][~m] == 0).all()
    values = oracle.value_forward(b.hidden, b.w_value) if cfg.value_head else b.values
    adv, ret, N = oracle.advantage(values, b.rewards, b.mask, b.cu_seqlens, cfg.gamma, cfg.lam, cfg.alpha)
    assert int(got["n"][0]) == N
    assert (np.abs(got["adv"] - adv) <= TOL_ADV * np.maximum(1, np.abs(adv))).all()
    assert (np.abs(got["ret"] - ret) <= TOL_ADV * np.maximum(1, np.abs(ret))).all()
    lro = rollout_logprobs(ref_lp, b.xi)
    loss, g, flags, counts = oracle.dis_loss(ref_lp, lro, adv, b.mask, cfg.eps_low, cfg.eps_high, N)
    assert np.array_equal(got["flags"], flags)
    assert np.array_equal(got["counts"], counts)
    check_loss(got, dict(loss=loss, flags=flags), ref_lp, lro, adv, b.mask, N)
    assert (np.abs(got["g"] - g) <= TOL_G * np.abs(g) + 1e-12).all()
    say(f"{name}: forward ok, clipped {counts[2] + counts[3]} of {counts[0]}")
    rng = np.random.default_rng(seed)
    if cfg.value_head:
        lv, dhv, dwv = oracle.value_loss(b.hidden, b.w_value, values, ret, b.mask, N)
        vrow = np.sort(rng.choice(np.nonzero(b.mask)[0], size=n_rows, replace=False))
        check_value(got, dict(v=values, lv=lv, dhv=dhv, dwv=dwv), b.mask, rows=vrow)
        del dhv
        say(f"{name}: critic ok")
    if not backward:
        return
    live = np.nonzero(g)[0]
    rows = np.sort(rng.choice(live, size=n_rows, replace=False))
    vrows = np.unique(np.concatenate([b.target[rows[:n_rows // 2]], rng.choice(cfg.V, n_rows, replace=False),
                                      [0, cfg.V - 1]]))
    w64 = b.w_head.astype(np.float64)
    if every_row:
        say(f"{name}: oracle backward on all {live.size} token rows with g != 0 and all {cfg.V} vocabulary rows")
        dH, dW = _oracle_backward_every_row(b, ref_lse, g, w64)
        check_grad(got["dh"], dH, np.nonzero(g == 0)[0], "dhidden (every row)")
        check_grad(got["dw"], dW, None, "dw_head (every row)")
        del dH, dW
    else:
        say(f"{name}: oracle backward on {rows.size} token rows and {vrows.size} vocabulary rows")
        dH, dW = oracle.loss_backward(b.hidden, None, b.target, ref_lse, g, dh_rows=rows, dw_rows=vrows, w64=w64)
        check_grad(got["dh"][rows], dH[rows], None, "dhidden rows")
        check_grad(got["dw"][vrows], dW[vrows], None, "dw_head rows")
    assert (got["dh"][g == 0] == 0).all()
    # the vocabulary sum of dz is 0 for every token, so sum_v dW_v = 0 up to rounding
    col = got["dw"].astype(np.float64).sum(axis=0)
    assert np.abs(col).max() <= 1e-2 * np.abs(got["dw"]).sum(axis=0).max()
    say(f"{name}: backward ok")


@pytest.mark.parametrize("name", ["c2", "c4"])
def test_loss_kernel_alone_on_oracle_logprobs(name):
    """sao_clipped_loss fed the oracle's own log-probs (rounded to fp32, as the
    library receives them): the loss kernel alone, without the head's log-prob
    error, against oracle.dis_loss on the same fp32 inputs. Flags and counts
    bit-exact; loss within 1e-5 of (1/N) sum |terms| and g within 1e-5 relative
    (the kernel's weight rho is evaluated in fp32)."""
    import os
    import paper_2607_07508_amd as sao
    if not os.path.exists(path_for(name)):
        pytest.skip("stored oracle values missing")
    cfg = CONFIGS[name]
    b = generate(cfg)
    ref_lp, _ = load_golden(name, b)
    lp32 = ref_lp.astype(np.float32)
    lro32 = rollout_logprobs(ref_lp, b.xi).astype(np.float32)
    values = oracle.value_forward(b.hidden, b.w_value) if cfg.value_head else b.values
    adv = oracle.advantage(values, b.rewards, b.mask, b.cu_seqlens, cfg.gamma, cfg.lam,
                           cfg.alpha)[0].astype(np.float32)
    N = int(b.mask.sum())
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    n_dev = torch.tensor([N], dtype=torch.int64, device="cuda")
    loss, g, flags, counts = sao.clipped_loss(t(lp32), t(lro32), t(adv), t(b.mask), cfg.eps_low, cfg.eps_high,
                                              n_dev)
    torch.cuda.synchronize()
    rl, rg, rf, rc = oracle.dis_loss(lp32, lro32, adv, b.mask, cfg.eps_low, cfg.eps_high, N)
    assert np.array_equal(flags.cpu().numpy(), rf)
    assert np.array_equal(counts.cpu().numpy(), rc)
    used = rf == 1
    lp64, rho = lp32.astype(np.float64), np.exp(lp32.astype(np.float64) - lro32)
    scale = (np.abs(rho * adv * lp64)[used].sum() / N, np.abs(rho * adv)[used].sum() / N)
    got = loss.cpu().numpy()
    for k in range(2):
        assert abs(got[k] - rl[k]) <= 1e-5 * max(abs(rl[k]), scale[k]), (k, got[k], rl[k])
    assert (np.abs(g.cpu().numpy() - rg) <= 1e-5 * np.abs(rg) + 1e-15).all()
    say(f"{name}: loss kernel alone ok, clipped {rc[2] + rc[3]} of {rc[0]}")


@pytest.mark.skipif(not __import__("os").path.exists(path_for("c2")), reason="stored oracle values missing")
def test_c2_full_forward_backward():
    # every dH and dW element against the oracle (a few minutes of fp64 BLAS on the host)
    _full("c2", backward=True, every_row=True)


@pytest.mark.skipif(not __import__("os").path.exists(path_for("c1")), reason="stored oracle values missing")
def test_c1_full_forward():
    _full("c1", backward=False)


@pytest.mark.skipif(not __import__("os").path.exists(path_for("c4")), reason="stored oracle values missing")
def test_c4_full_forward_backward_value_head():
    _full("c4", backward=True)


@pytest.mark.skipif(not __import__("os").path.exists(path_for("c3")), reason="stored oracle values missing")
def test_c3_full_chunked_forward_backward():
    _full("c3", backward=True)
