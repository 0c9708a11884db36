"""GPU parity of the whole hot path (through the C ABI) against the fp64 oracle.

Sizes span several tiles with ragged tails, several vocabulary blocks of the
backward, fp32 and bf16, and the degenerate cases (single token, all masked,
minimum H, target out of range, malformed segments).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_07508_amd as sao
from synth import CONFIGS, bf16_bits, bf16_round, generate, small_config, with_overrides
from synth.device import to_device
from tests.gpu_common import (TOL_LOGP, TOL_LOSS, TOL_V, check_grad, compare_all, gpu_pass, oracle_pass, say)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    sao.lib()


def _roundtrip(cfg, gamma=1.0, lam=1.0, alpha=0.0, backward=True):
    say(f"case {cfg.name}: T={cfg.T} H={cfg.H} V={cfg.V} {cfg.dtype} gamma={gamma} lam={lam} alpha={alpha}")
    b = generate(cfg)
    ref = oracle_pass(b, gamma, lam, alpha, backward)
    got = gpu_pass(b, ref["logp"], gamma, lam, alpha, backward)
    compare_all(got, ref, b, backward)
    say(f"case {cfg.name}: ok (clipped {ref['counts'][2] + ref['counts'][3]} of {ref['counts'][0]})")
    return got, ref


def test_c0_fp32_fixed_lambda():
    _roundtrip(CONFIGS["c0"], 1.0, 1.0, 0.0)


def test_c0_fp32_length_adaptive():
    _roundtrip(CONFIGS["c0"], 1.0, 1.0, 1.5)


def test_c0_as_bf16():
    _roundtrip(with_overrides(CONFIGS["c0"], name="c0-bf16", dtype="bf16"), 0.99, 0.95, 0.0)


@pytest.mark.parametrize("case", [
    dict(name="m1", seed=11, B=5, T=700, H=192, V=2000),            # 8 vocab tiles, ragged tails
    dict(name="m2", seed=12, B=3, T=300, H=64, V=1001),             # V not a multiple of 8
    dict(name="m3", seed=13, B=4, T=640, H=64, V=140000),           # three backward vocab blocks
    dict(name="m4", seed=14, B=2, T=50, H=8, V=300),                # minimum H
    dict(name="m5", seed=15, B=6, T=1100, H=320, V=520, dtype="f32"),
])
def test_mid_sizes(case):
    cfg = small_config(**case)
    _roundtrip(cfg, 1.0, 1.0, 1.5)


def test_single_token():
    cfg = small_config("one", 21, B=1, T=1, H=16, V=77, act_span=(1, 1), obs_span=(1, 1))
    _roundtrip(cfg)


def test_peaked_logits():
    # hidden and W ~ N(0, 1) at H = 64: logits of std 8, near one-hot softmax
    cfg = small_config("peaked", 22, B=3, T=400, H=64, V=3000, init_std=1.0, dtype="f32")
    _roundtrip(cfg, 0.99, 0.9)
    cfg = small_config("peaked-bf16", 23, B=3, T=400, H=64, V=3000, init_std=1.0)
    _roundtrip(cfg, 0.99, 0.9)


def test_all_masked_and_zero_gradient():
    b = generate(small_config("masked", 24, B=2, T=300, H=64, V=500))
    b.mask[:] = 0
    db = to_device(b, np.zeros(b.T))
    logp, lse = sao.token_logprob(db.hidden, db.w_head, db.target, db.mask)
    adv, ret, n = sao.advantage(db.values, db.rewards, db.mask, db.cu_seqlens, 1.0, 1.0, 0.0)
    loss, g, flags, counts = sao.clipped_loss(logp, db.logp_rollout, adv, db.mask, 0.2, 0.2, n)
    dw0 = torch.full((b.cfg.V, b.cfg.H), 0.5, dtype=torch.float32, device="cuda")
    dh, dw = sao.loss_backward(db.hidden, db.w_head, db.target, lse, g, dw_head=dw0)
    torch.cuda.synchronize()
    assert (logp == 0).all() and (lse == 0).all() and (adv == 0).all() and int(n) == 0
    assert (loss == 0).all() and (counts == 0).all() and (g == 0).all() and (flags == 0).all()
    assert (dh == 0).all() and (dw == 0.5).all()


def test_accumulation_and_determinism():
    b = generate(small_config("acc", 25, B=4, T=900, H=128, V=1500))
    ref = oracle_pass(b, 1.0, 1.0, 1.5)
    db = to_device(b, ref["logp"])
    runs = []
    for _ in range(2):
        logp, lse = sao.token_logprob(db.hidden, db.w_head, db.target, db.mask)
        adv, ret, n = sao.advantage(db.values, db.rewards, db.mask, db.cu_seqlens, 1.0, 1.0, 1.5)
        loss, g, flags, counts = sao.clipped_loss(logp, db.logp_rollout, adv, db.mask, 0.2, 0.2, n)
        # a second call accumulates into loss / counts
        sao.clipped_loss(logp, db.logp_rollout, adv, db.mask, 0.2, 0.2, n, loss=loss, counts=counts)
        dh, dw = sao.loss_backward(db.hidden, db.w_head, db.target, lse, g)
        sao.loss_backward(db.hidden, db.w_head, db.target, lse, g, dw_head=dw)
        torch.cuda.synchronize()
        runs.append([x.cpu().float().numpy() for x in (logp, loss, flags, counts, dh, dw)])
    for a, c in zip(runs[0], runs[1]):
        assert np.array_equal(a, c)
    logp, loss, flags, counts, dh, dw = runs[0]
    assert np.array_equal(counts, 2 * ref["counts"])
    assert np.allclose(loss, 2 * ref["loss"], rtol=1e-3, atol=0)
    check_grad(dw, 2 * ref["dw"], None, "dw x2")


def test_forward_launch_forms_agree():
    """Up to 8192 tokens the forward runs one workgroup per CU pulling tiles; above
    it, one workgroup per tile. Both compute every tile's log-sum-exp partials the
    same way and merge them in the same order, so the first 8192 rows come out
    bit for bit the same either way; sampled rows match the oracle."""
    T, H, V = 8193, 64, 3000
    b = generate(small_config("launch-forms", 27, B=8, T=T, H=H, V=V))
    hid = torch.from_numpy(bf16_bits(b.hidden)).view(torch.bfloat16).cuda()
    w = torch.from_numpy(bf16_bits(b.w_head)).view(torch.bfloat16).cuda()
    tgt = torch.from_numpy(b.target).cuda()
    mask = torch.from_numpy(b.mask).cuda()
    say(f"case launch-forms: T={T} (tiles pulled) and {T - 1} (one workgroup per tile), H={H} V={V}")
    lp_a, lse_a = sao.token_logprob(hid, w, tgt, mask)                       # 8193 rows: one workgroup per tile
    lp_b, lse_b = sao.token_logprob(hid[:T - 1], w, tgt[:T - 1], mask[:T - 1])  # 8192 rows: pulled
    torch.cuda.synchronize()
    assert torch.equal(lp_a[:T - 1], lp_b) and torch.equal(lse_a[:T - 1], lse_b)
    rows = np.nonzero(b.mask)[0][::97]
    ref_lp, ref_lse = oracle.token_logprob(b.hidden, b.w_head, b.target, rows=rows)
    assert np.abs(lp_b.cpu().numpy()[rows] - ref_lp[rows]).max() <= TOL_LOGP
    assert np.abs(lse_b.cpu().numpy()[rows] - ref_lse[rows]).max() <= TOL_LOGP


def test_chunked_equals_whole():
    """Token chunks with the global N: losses, counts and dW sum to the whole-batch values."""
    b = generate(small_config("chunks", 26, B=3, T=1200, H=64, V=900))
    ref = oracle_pass(b, 1.0, 1.0, 1.5)
    db = to_device(b, ref["logp"])
    adv, ret, n = sao.advantage(db.values, db.rewards, db.mask, db.cu_seqlens, 1.0, 1.0, 1.5)
    loss = torch.zeros(2, dtype=torch.float64, device="cuda")
    counts = torch.zeros(5, dtype=torch.int64, device="cuda")
    dw = torch.zeros((b.cfg.V, b.cfg.H), dtype=torch.float32, device="cuda")
    dh = torch.empty_like(db.hidden)
    for s in range(0, b.T, 256):
        e = min(s + 256, b.T)
        lp, lse = sao.token_logprob(db.hidden[s:e], db.w_head, db.target[s:e], db.mask[s:e])
        _, g, _, _ = sao.clipped_loss(lp, db.logp_rollout[s:e], adv[s:e], db.mask[s:e], 0.2, 0.2, n,
                                      loss=loss, counts=counts)
        sao.loss_backward(db.hidden[s:e], db.w_head, db.target[s:e], lse, g, dw_head=dw, dhidden=dh[s:e])
    torch.cuda.synchronize()
    assert np.array_equal(counts.cpu().numpy(), ref["counts"])
    assert np.allclose(loss.cpu().numpy(), ref["loss"], rtol=1e-3, atol=1e-12)
    check_grad(dw.cpu().numpy(), ref["dw"], None, "chunked dw")
    check_grad(dh.float().cpu().numpy(), ref["dh"], np.nonzero(ref["g"] == 0)[0], "chunked dh")


def test_target_out_of_range_sets_status():
    b = generate(small_config("badtgt", 27, B=2, T=200, H=64, V=400))
    t_bad = int(np.nonzero(b.mask)[0][3])
    b.target[t_bad] = b.cfg.V
    db = to_device(b)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    logp, lse = sao.token_logprob(db.hidden, db.w_head, db.target, db.mask, status=status)
    torch.cuda.synchronize()
    assert int(status) & sao.binding.STATUS_TARGET_RANGE
    lp = logp.cpu().numpy()
    assert np.isnan(lp[t_bad])
    ok = (b.mask == 1) & (np.arange(b.T) != t_bad)
    ref, _ = oracle.token_logprob(b.hidden, b.w_head, np.minimum(b.target, b.cfg.V - 1), b.mask)
    assert np.abs(lp[ok] - ref[ok]).max() <= TOL_LOGP


@pytest.mark.parametrize("bad", [np.nan, np.inf])
def test_nonfinite_hidden_sets_status(bad):
    # a non-finite hidden state makes its row's log-sum-exp non-finite: the row's
    # log-prob is not finite, the status word gets the non-finite bit, and every
    # other row is unaffected
    b = generate(small_config("badh", 29, B=2, T=300, H=64, V=700, dtype="f32"))
    t_bad = int(np.nonzero(b.mask)[0][5])
    ref, _ = oracle.token_logprob(b.hidden, b.w_head, b.target, b.mask)
    b.hidden[t_bad, 7] = bad
    db = to_device(b)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    logp, lse = sao.token_logprob(db.hidden, db.w_head, db.target, db.mask, status=status)
    torch.cuda.synchronize()
    assert int(status) & sao.binding.STATUS_NONFINITE
    assert not (int(status) & sao.binding.STATUS_TARGET_RANGE)
    lp, ls = logp.cpu().numpy(), lse.cpu().numpy()
    assert not np.isfinite(ls[t_bad]) and not np.isfinite(lp[t_bad])
    ok = (b.mask == 1) & (np.arange(b.T) != t_bad)
    assert np.isfinite(lp[ok]).all()
    assert np.abs(lp[ok] - ref[ok]).max() <= TOL_LOGP


def test_malformed_segments_set_status():
    b = generate(small_config("badcu", 28, B=3, T=120, H=8, V=16))
    db = to_device(b)
    cu_np = b.cu_seqlens.copy()
    cu_np[1], cu_np[2] = cu_np[2], cu_np[1]       # a decreasing boundary
    assert cu_np[2] < cu_np[1]
    cu = torch.from_numpy(cu_np).cuda()
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    adv, ret, n = sao.advantage(db.values, db.rewards, db.mask, cu, 1.0, 1.0, 0.0, status=status)
    torch.cuda.synchronize()
    assert int(status) & sao.binding.STATUS_SEGMENTS
    assert np.isnan(adv.cpu().numpy()).any()


@pytest.mark.parametrize("case", [
    dict(name="v1", seed=31, B=4, T=900, H=320, V=700, value_head=True),
    dict(name="v2", seed=32, B=3, T=500, H=72, V=300, dtype="f32", value_head=True),      # H % 32 != 0
    dict(name="v3", seed=33, B=8, T=2500, H=512, V=4000, eps_high=0.28, value_head=True),  # c4's shape mix
])
def test_value_head(case):
    """Critic values feed the scan; its squared-error loss and gradients."""
    _roundtrip(small_config(**case), 1.0, 1.0, 1.5)


def test_value_loss_local_count_and_masked_rows():
    b = generate(small_config("vmask", 34, B=3, T=600, H=96, V=200, value_head=True))
    b.mask[:200] = 0
    ref = oracle_pass(b, 1.0, 1.0, 1.5, backward=False)
    db = to_device(b, ref["logp"])
    v = sao.value_forward(db.hidden, db.w_value)
    adv, ret, n = sao.advantage(v, db.rewards, db.mask, db.cu_seqlens, 1.0, 1.0, 1.5)
    lv_g, dh_g, dw_g = sao.value_loss(db.hidden, db.w_value, v, ret, db.mask, n)
    lv_l, dh_l, dw_l = sao.value_loss(db.hidden, db.w_value, v, ret, db.mask, None)   # N = sum(mask)
    # a second call accumulates into the loss and dw_v
    sao.value_loss(db.hidden, db.w_value, v, ret, db.mask, n, loss=lv_g, dw_value=dw_g)
    torch.cuda.synchronize()
    assert torch.equal(dh_g, dh_l) and (dh_g[:200] == 0).all()
    assert abs(float(lv_g) - 2 * float(lv_l)) <= 1e-12 * abs(float(lv_l))
    assert abs(float(lv_l) - ref["lv"]) <= TOL_LOSS * abs(ref["lv"])
    check_grad(dw_g.cpu().numpy()[None, :], 2 * ref["dwv"][None, :], None, "dw_v x2")
    assert (np.abs(v.cpu().numpy() - ref["v"]) <= TOL_V * np.maximum(1, np.abs(ref["v"]))).all()


def test_value_loss_all_masked():
    b = generate(small_config("vzero", 35, B=2, T=300, H=64, V=100, value_head=True))
    b.mask[:] = 0
    db = to_device(b)
    v = sao.value_forward(db.hidden, db.w_value)
    ret = torch.randn(b.T, device="cuda")
    dw0 = torch.full((b.cfg.H,), 0.25, dtype=torch.float32, device="cuda")
    lv, dh, dw = sao.value_loss(db.hidden, db.w_value, v, ret, db.mask, None, dw_value=dw0)
    torch.cuda.synchronize()
    assert float(lv) == 0.0 and (dh == 0).all() and (dw == 0.25).all()


def test_value_dhidden_is_rne_of_fp32_product():
    """dH_v = bf16(dv * w_v): the kernel's fp32 product rounded to nearest even, bit for bit."""
    b = generate(small_config("vrne", 36, B=3, T=700, H=256, V=100, value_head=True))
    db = to_device(b)
    rng = np.random.default_rng(36)
    ret_h = rng.normal(0.5, 0.5, b.T).astype(np.float32)
    v = sao.value_forward(db.hidden, db.w_value)
    _, dh, _ = sao.value_loss(db.hidden, db.w_value, v, torch.from_numpy(ret_h).cuda(), db.mask, None)
    torch.cuda.synchronize()
    m = b.mask != 0
    N = int(m.sum())
    d64 = v.cpu().numpy().astype(np.float64) - ret_h.astype(np.float64)
    dv = np.where(m, (2.0 * d64 * (1.0 / N)).astype(np.float32), np.float32(0.0))
    prod = dv[:, None] * b.w_value[None, :].astype(np.float32)
    want = bf16_bits(bf16_round(prod))
    want[~m] = 0
    got = dh.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, want), int((got != want).sum())


@pytest.mark.parametrize("eps_low,eps_high", [(0.2, 0.28), (0.3, 5.0), (0.8, 3.0)])
def test_band_decisions_near_edges(eps_low, eps_high):
    """Ratios within 1e-6 of either band edge (in log space) flag exactly as in float64."""
    rng = np.random.default_rng(41)
    n = 8192
    lro = rng.uniform(-6.0, -0.05, n).astype(np.float32)
    edges = np.array([np.log1p(-eps_low), np.log1p(eps_high)])
    d = edges[rng.integers(0, 2, n)] + rng.uniform(-1e-6, 1e-6, n)
    lp = (lro.astype(np.float64) + d).astype(np.float32)
    adv = rng.normal(0.0, 1.0, n).astype(np.float32)
    mask = np.ones(n, dtype=np.uint8)
    mask[::17] = 0
    t = lambda x: torch.from_numpy(x).cuda()  # noqa: E731
    loss, g, flags, counts = sao.clipped_loss(t(lp), t(lro), t(adv), t(mask), eps_low, eps_high, None)
    torch.cuda.synchronize()
    ref_loss, ref_g, ref_flags, ref_counts = oracle.dis_loss(lp.astype(np.float64), lro.astype(np.float64), adv,
                                                             mask, eps_low, eps_high)
    assert np.array_equal(flags.cpu().numpy(), ref_flags)
    assert np.array_equal(counts.cpu().numpy(), ref_counts)
    assert ref_counts[2] > 100 and ref_counts[3] > 100 and ref_counts[1] > 100
    assert np.allclose(loss.cpu().numpy(), ref_loss, rtol=1e-5, atol=1e-12)
    assert np.allclose(g.cpu().numpy(), ref_g, rtol=1e-5, atol=1e-12)


def test_band_without_lower_edge_and_extremes():
    """eps_low >= 1 clips low only where exp underflows; +-inf and NaN ratios."""
    lp = np.array([-800.0, -0.5, 0.0, -3.0, np.inf, -np.inf, np.nan, -1.0], dtype=np.float32)
    lro = np.array([0.0, 0.0, 0.0, -3.0, 0.0, 0.0, 0.0, np.nan], dtype=np.float32)
    adv = np.linspace(-1.0, 1.0, lp.size).astype(np.float32)
    mask = np.ones(lp.size, dtype=np.uint8)
    t = lambda x: torch.from_numpy(x).cuda()  # noqa: E731
    for eps_low in (1.0, 1.5, 0.2):
        loss, g, flags, counts = sao.clipped_loss(t(lp), t(lro), t(adv), t(mask), eps_low, 0.28, None)
        torch.cuda.synchronize()
        rl, rg, rf, rc = oracle.dis_loss(lp.astype(np.float64), lro.astype(np.float64), adv, mask, eps_low, 0.28)
        assert np.array_equal(flags.cpu().numpy(), rf), (eps_low, flags.cpu().numpy(), rf)
        assert np.array_equal(counts.cpu().numpy(), rc)
        # with eps_low = 1.5 the band's lower edge is 0, so the log pi = -inf token
        # (rho = 0) is clipped low and the loss stays finite
        assert np.isfinite(rl).all()
        assert np.allclose(loss.cpu().numpy(), rl, rtol=1e-5, atol=1e-12)


def test_seven_row_vocabulary():
    """A head of seven rows: a single, mostly empty vocabulary tile."""
    _roundtrip(small_config("v7", 67, B=3, T=500, H=64, V=7), 1.0, 1.0, 1.5)


def test_one_row_vocabulary():
    """With V = 1, log pi = 0 and dz = g (1 - p) = 0 exactly: both sides hold only
    rounding there, so those are checked against their natural scale."""
    from tests.gpu_common import check_loss
    b = generate(small_config("v1", 61, B=3, T=500, H=64, V=1))
    ref = oracle_pass(b, 1.0, 1.0, 1.5)
    got = gpu_pass(b, ref["logp"], 1.0, 1.0, 1.5)
    m = b.mask == 1
    assert np.abs(got["logp"][m]).max() <= 1e-6 and (got["logp"][~m] == 0).all()
    assert np.array_equal(got["flags"], ref["flags"]) and np.array_equal(got["counts"], ref["counts"])
    check_loss(got, ref, ref["logp"], ref["lro"], ref["adv"], b.mask, ref["n"], propagated_floor=True)
    gmax = np.abs(ref["g"]).max()
    assert np.abs(got["dh"]).max() <= 1e-5 * gmax * np.abs(b.w_head).max()
    assert np.abs(got["dw"]).max() <= 1e-5 * gmax * np.abs(b.hidden).sum(axis=0).max()


def _scan_case(name, seed, B, T, cu=None, mask_fn=None):
    b = generate(small_config(name, seed, B=B, T=T, H=8, V=16))
    if cu is not None:
        b.cu_seqlens[:] = np.asarray(cu, dtype=np.int32)
    if mask_fn is not None:
        mask_fn(b)
    adv_r, ret_r, n_r = oracle.advantage(b.values, b.rewards, b.mask, b.cu_seqlens, 0.99, 0.9, 1.5)
    return b, adv_r, ret_r, n_r


def _check_scan(got, adv_r, ret_r, n_r):
    adv, ret, n = (x.cpu().numpy() for x in got)
    assert int(n[0]) == n_r
    assert (np.abs(adv - adv_r) <= 1e-6 * np.maximum(1, np.abs(adv_r))).all()
    assert (np.abs(ret - ret_r) <= 1e-6 * np.maximum(1, np.abs(ret_r))).all()


def test_scan_empty_and_observation_only_trajectories():
    T = 5000
    cu = [0, 0, 1200, 1200, 1201, 3300, 3300, T]          # empty segments, a one-token one
    def obs_only(b):
        b.mask[1201:3300] = 0                              # a trajectory with no action at all
        b.rewards[1201:3300] = 0.25
    b, a, r, n = _scan_case("scan-edge", 71, B=7, T=T, cu=cu, mask_fn=obs_only)
    db = to_device(b)
    got = sao.advantage(db.values, db.rewards, db.mask, db.cu_seqlens, 0.99, 0.9, 1.5)
    torch.cuda.synchronize()
    _check_scan(got, a, r, n)


def test_scan_one_long_trajectory():
    """One trajectory over many 2048-token tiles, ending mid-tile."""
    T = 70001
    b, a, r, n = _scan_case("scan-long", 72, B=1, T=T, cu=[0, T])
    db = to_device(b)
    got = sao.advantage(db.values, db.rewards, db.mask, db.cu_seqlens, 0.99, 0.9, 1.5)
    torch.cuda.synchronize()
    _check_scan(got, a, r, n)


@pytest.mark.parametrize("gamma,lam", [(0.0, 0.0), (0.0, 1.0), (1.0, 0.0), (1.0, 1.0)])
def test_scan_degenerate_discounts(gamma, lam):
    """gamma and lambda at 0 and 1 (fixed lambda): the scan's composed maps then carry
    zero or unit coefficients through many tiles; rewards also sit on observations."""
    T = 40000
    cu = [0, 9000, 9001, 26000, 26000, T]                 # multi-tile, one-token and empty trajectories
    def obs_rewards(b):
        obs = b.mask == 0
        b.rewards[obs] = np.random.default_rng(73).normal(0.0, 0.5, int(obs.sum())).astype(np.float32)
    b = generate(small_config("scan-deg", 74, B=5, T=T, H=8, V=16))
    b.cu_seqlens[:] = np.asarray(cu, dtype=np.int32)
    obs_rewards(b)
    a, r, n = oracle.advantage(b.values, b.rewards, b.mask, b.cu_seqlens, gamma, lam, 0.0)
    db = to_device(b)
    got = sao.advantage(db.values, db.rewards, db.mask, db.cu_seqlens, gamma, lam, 0.0)
    torch.cuda.synchronize()
    _check_scan(got, a, r, n)


def test_unaligned_per_token_arrays():
    """Slices at odd offsets take the scalar paths of the scan and the loss."""
    b = generate(small_config("unaligned", 73, B=5, T=3001, H=64, V=200))
    ref = oracle_pass(b, 0.99, 0.9, 1.5, backward=False)
    db = to_device(b, ref["logp"])
    # copy every per-token array into a buffer one element longer and take [1:]
    def shifted(x):
        buf = torch.empty(x.numel() + 1, dtype=x.dtype, device=x.device)
        buf[1:] = x
        return buf[1:]
    vals, rews, mask = shifted(db.values), shifted(db.rewards), shifted(db.mask)
    assert vals.data_ptr() % 16 != 0 and mask.data_ptr() % 8 != 0
    adv, ret, n = sao.advantage(vals, rews, mask, db.cu_seqlens, 0.99, 0.9, 1.5)
    _check_scan((adv, ret, n), ref["adv"], ref["ret"], ref["n"])
    lp = shifted(torch.from_numpy(ref["logp"].astype(np.float32)).cuda())
    lro = shifted(db.logp_rollout)
    loss, g, flags, counts = sao.clipped_loss(lp, lro, shifted(torch.from_numpy(ref["adv"].astype(np.float32)).cuda()),
                                              mask, b.cfg.eps_low, b.cfg.eps_high, n)
    torch.cuda.synchronize()
    assert np.array_equal(flags.cpu().numpy(), ref["flags"])
    assert np.array_equal(counts.cpu().numpy(), ref["counts"])
    assert np.allclose(loss.cpu().numpy(), ref["loss"], rtol=1e-5, atol=1e-12)



def test_backward_operand_past_4gib():
    # About 150k token rows reach the backward, so its bf16 dz scratch (rows x
    # 16384 vocabulary entries) spans 4.9 GB and the dH product reads a K-major
    # operand past the reach of a 32-bit byte offset from the operand's start.
    # Both sides get the same seeded g; the oracle recomputes lse and dH for
    # sampled rows, taken mostly past compacted row 131072.
    T, H, V = 150000, 64, 16384
    cfg = small_config("dz-past-4gib", 41, B=16, T=T, H=H, V=V, act_span=(64, 400), obs_span=(1, 4))
    b = generate(cfg)
    rng = np.random.default_rng(41)
    g = (rng.standard_normal(T) / T).astype(np.float32)
    g[rng.random(T) < 0.01] = 0.0
    say(f"case dz-past-4gib: T={T} H={H} V={V}, {int((g != 0).sum())} backward rows")
    assert int((g != 0).sum()) * V * 2 > 2**32
    dev = "cuda"
    hid = torch.from_numpy(bf16_bits(b.hidden)).view(torch.bfloat16).to(dev)
    w = torch.from_numpy(bf16_bits(b.w_head)).view(torch.bfloat16).to(dev)
    tgt = torch.from_numpy(b.target).to(dev)
    _, lse = sao.token_logprob(hid, w, tgt)
    dh, dw = sao.loss_backward(hid, w, tgt, lse, torch.from_numpy(g).to(dev))
    torch.cuda.synchronize()
    live = np.nonzero(g)[0]
    rows = np.sort(np.concatenate([rng.choice(live[live.size * 9 // 10:], 20, replace=False),
                                   rng.choice(live[:live.size * 9 // 10], 4, replace=False)]))
    say(f"case dz-past-4gib: oracle on {rows.size} rows, compacted indices up to {int(np.searchsorted(live, rows[-1]))}")
    ref_lp, ref_lse = oracle.token_logprob(b.hidden, b.w_head, b.target, rows=rows)
    got_lse = lse.cpu().numpy()
    assert np.abs(got_lse[rows] - ref_lse[rows]).max() <= TOL_LOGP
    ref_dh, _ = oracle.loss_backward(b.hidden, b.w_head, b.target, ref_lse, g, dh_rows=rows, dw_rows=[])
    got_dh = dh.float().cpu().numpy()
    check_grad(got_dh[rows], ref_dh[rows], None, "dhidden rows past 4 GiB")
    assert (got_dh[g == 0] == 0).all()
    say("case dz-past-4gib: ok")


def _padded(x: np.ndarray, pad: int, dtype: str) -> torch.Tensor:
    """The rows of x in a device buffer whose rows are `pad` elements longer (a strided view)."""
    rows, cols = x.shape
    if dtype == "bf16":
        buf = torch.zeros(rows, cols + pad, dtype=torch.bfloat16)
        buf[:, :cols] = torch.from_numpy(bf16_bits(x)).view(torch.bfloat16)
    else:
        buf = torch.zeros(rows, cols + pad, dtype=torch.float32)
        buf[:, :cols] = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return buf.to("cuda")[:, :cols]


@pytest.mark.parametrize("dtype,H,pad_h,pad_w", [("bf16", 192, 24, 40), ("f32", 96, 8, 32)])
def test_padded_leading_dimensions(dtype, H, pad_h, pad_w):
    # hidden and W_head rows with leading dimensions above H: the forward reads
    # both K-major, the backward reads W MN-major and gathers hidden rows, and
    # the critic reads hidden rows.
    cfg = small_config(f"ld-{dtype}", 51, B=3, T=700, H=H, V=2000, dtype=dtype, value_head=True)
    b = generate(cfg)
    say(f"case ld-{dtype}: H={H} ld_hidden={H + pad_h} ld_w={H + pad_w}")
    rng = np.random.default_rng(51)
    g = np.where((b.mask == 1) & (rng.random(b.T) < 0.7), rng.standard_normal(b.T) / b.T, 0.0).astype(np.float32)
    ref_lp, ref_lse = oracle.token_logprob(b.hidden, b.w_head, b.target, b.mask)
    ref_dh, ref_dw = oracle.loss_backward(b.hidden, b.w_head, b.target, ref_lse, g)
    ref_v = oracle.value_forward(b.hidden, b.w_value)
    hid, w = _padded(b.hidden, pad_h, dtype), _padded(b.w_head, pad_w, dtype)
    assert hid.stride(0) == H + pad_h and w.stride(0) == H + pad_w
    tgt = torch.from_numpy(b.target).cuda()
    mask = torch.from_numpy(b.mask).cuda()
    logp, lse = sao.token_logprob(hid, w, tgt, mask)
    all_lse = sao.token_logprob(hid, w, tgt)[1]
    dh, dw = sao.loss_backward(hid, w, tgt, all_lse, torch.from_numpy(g).cuda())
    wv = torch.from_numpy(bf16_bits(b.w_value)).view(torch.bfloat16) if dtype == "bf16" else \
        torch.from_numpy(np.ascontiguousarray(b.w_value, dtype=np.float32))
    v = sao.value_forward(hid, wv.cuda())
    torch.cuda.synchronize()
    m = b.mask == 1
    assert np.abs(logp.cpu().numpy()[m] - ref_lp[m]).max() <= TOL_LOGP
    assert np.abs(lse.cpu().numpy()[m] - ref_lse[m]).max() <= TOL_LOGP
    check_grad(dh.float().cpu().numpy(), ref_dh, np.nonzero(g == 0)[0], "dhidden")
    check_grad(dw.cpu().numpy(), ref_dw, None, "dw_head")
    got_v = v.cpu().numpy()
    assert (np.abs(got_v - ref_v) <= TOL_V * np.maximum(1.0, np.abs(ref_v))).all()
    say(f"case ld-{dtype}: ok")


def test_side_stream_matches_default_stream():
    # Every launch goes on the caller's current stream: the same calls on a
    # side stream (default priority) give bit-identical results.
    b = generate(small_config("stream", 61, B=3, T=900, H=128, V=3000))
    db = to_device(b)
    rng = np.random.default_rng(61)
    g = torch.from_numpy(np.where(b.mask == 1, rng.standard_normal(b.T) / b.T, 0.0).astype(np.float32)).cuda()

    def run():
        logp, lse = sao.token_logprob(db.hidden, db.w_head, db.target, db.mask)
        all_lse = sao.token_logprob(db.hidden, db.w_head, db.target)[1]
        dh, dw = sao.loss_backward(db.hidden, db.w_head, db.target, all_lse, g)
        return logp, lse, dh, dw

    ref = run()
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        got = run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for a, c in zip(ref, got):
        assert torch.equal(a, c)
