"""Shared helpers of the GPU parity tests: run the HIP path and the oracle, compare.

Tolerances (the GPU side computes in fp32 from bf16/fp32 inputs; the oracle in fp64):
  log-probs and lse: max abs <= 2e-3 (expected ~1e-5)
  flags, counts, N: bit-exact (the drift noise keeps every ratio >= 4e-3 in
      log space from a band edge, far beyond the ~1e-5 log-prob error)
  loss values: |d| <= 1e-3 * max(|ref|, (1/N) sum |terms|). Only the one-row
      vocabulary test (log pi exactly 0, so the reference loss is exactly 0 and
      both sides hold nothing but rounding) asks for a floor: 4x the change that
      the measured per-token log-prob differences propagate into the loss
  g: |d| <= 1e-3 * |ref| + 1e-12 (g = -rho A / N inherits the log-prob error ~1e-5)
  advantages/returns: |d| <= 1e-6 * max(1, |ref|) (fp64 inside, rounded to fp32)
  dH, dW: Frobenius relative <= 1e-2, per-row relative <= 1e-2 on rows whose norm
      exceeds 1e-3 of the largest row, rows with g = 0 exactly zero
  critic values v: |d| <= 1e-5 * max(1, |ref|) (fp32 accumulation over H products
      that are exact in fp32); L_V: relative 1e-3; dH_v, dw_v as dH, dW, rows with
      mask 0 exactly zero
"""
from __future__ import annotations

import sys
import time

import numpy as np
import torch

import oracle
import paper_2607_07508_amd as sao
from synth import rollout_logprobs
from synth.device import to_device

TOL_LOGP = 2e-3
TOL_LOSS = 1e-3
TOL_G = 1e-3
TOL_ADV = 1e-6
TOL_GRAD = 1e-2
TOL_V = 1e-5


def say(msg: str) -> None:
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def gpu_pass(batch, ref_logp, gamma, lam, alpha, backward=True, n_tokens_global=True, chunk=None,
             value_head=None):
    """The whole hot path on the GPU through the C ABI; returns host numpy results.

    With a critic head (the batch carries w_value; value_head=None follows it) the
    GAE values are the head's outputs and the squared-error loss runs after the
    scan. With `chunk`, the head passes run over token chunks of that size with
    the whole batch's N (the scan always covers the whole batch)."""
    cfg = batch.cfg
    db = to_device(batch, ref_logp)
    use_v = (db.w_value is not None) if value_head is None else value_head
    out = {}
    values = db.values
    if use_v:
        values = sao.value_forward(db.hidden, db.w_value)
        out["v"] = values
    adv, ret, n_tok = sao.advantage(values, db.rewards, db.mask, db.cu_seqlens, gamma, lam, alpha)
    out.update(adv=adv, ret=ret, n=n_tok)
    n_arg = n_tok if n_tokens_global else None
    T = batch.T
    step = T if not chunk else chunk
    dev = db.target.device
    logp = torch.empty(T, dtype=torch.float32, device=dev)
    lse = torch.empty_like(logp)
    g = torch.empty_like(logp)
    flags = torch.empty(T, dtype=torch.uint8, device=dev)
    loss = torch.zeros(2, dtype=torch.float64, device=dev)
    counts = torch.zeros(5, dtype=torch.int64, device=dev)
    dh = torch.empty_like(db.hidden) if backward else None
    dw = torch.zeros((cfg.V, cfg.H), dtype=torch.float32, device=dev) if backward else None
    for s in range(0, T, step):
        e = min(T, s + step)
        lp_c, lse_c = sao.token_logprob(db.hidden[s:e], db.w_head, db.target[s:e], db.mask[s:e])
        _, g_c, fl_c, _ = sao.clipped_loss(lp_c, db.logp_rollout[s:e], adv[s:e], db.mask[s:e], cfg.eps_low,
                                           cfg.eps_high, n_arg, loss=loss, counts=counts)
        logp[s:e], lse[s:e], g[s:e], flags[s:e] = lp_c, lse_c, g_c, fl_c
        if backward:
            sao.loss_backward(db.hidden[s:e], db.w_head, db.target[s:e], lse_c, g_c, dw_head=dw,
                              dhidden=dh[s:e])
    out.update(logp=logp, lse=lse, loss=loss, g=g, flags=flags, counts=counts)
    if backward:
        out.update(dh=dh, dw=dw)
    if use_v:
        lv, dhv, dwv = sao.value_loss(db.hidden, db.w_value, values, ret, db.mask, n_arg)
        out.update(lv=lv, dhv=dhv, dwv=dwv)
    torch.cuda.synchronize()
    res = {}
    for k, v in out.items():
        if v.dtype == torch.bfloat16:
            v = v.float()
        res[k] = v.cpu().numpy()
    return res


def oracle_pass(batch, gamma, lam, alpha, backward=True, value_head=None):
    cfg = batch.cfg
    use_v = (batch.w_value is not None) if value_head is None else value_head
    lp, lse = oracle.token_logprob(batch.hidden, batch.w_head, batch.target, batch.mask)
    values = oracle.value_forward(batch.hidden, batch.w_value) if use_v else batch.values
    adv, ret, N = oracle.advantage(values, batch.rewards, batch.mask, batch.cu_seqlens, gamma, lam, alpha)
    lro = rollout_logprobs(lp, batch.xi)
    loss, g, flags, counts = oracle.dis_loss(lp, lro, adv, batch.mask, cfg.eps_low, cfg.eps_high, N)
    res = dict(logp=lp, lse=lse, adv=adv, ret=ret, n=N, loss=loss, g=g, flags=flags, counts=counts, lro=lro)
    if backward:
        dh, dw = oracle.loss_backward(batch.hidden, batch.w_head, batch.target, lse, g)
        res.update(dh=dh, dw=dw)
    if use_v:
        lv, dhv, dwv = oracle.value_loss(batch.hidden, batch.w_value, values, ret, batch.mask, N)
        res.update(v=values, lv=lv, dhv=dhv, dwv=dwv)
    return res


def check_value(got, ref, mask, rows=None):
    """Critic outputs against the oracle (dH_v on `rows` only when given)."""
    assert (np.abs(got["v"] - ref["v"]) <= TOL_V * np.maximum(1.0, np.abs(ref["v"]))).all()
    lv_ref = float(ref["lv"])
    assert abs(float(got["lv"][0]) - lv_ref) <= TOL_LOSS * abs(lv_ref) + 1e-300, (got["lv"], lv_ref)
    check_grad(got["dwv"][None, :], np.asarray(ref["dwv"])[None, :], None, "dw_value")
    zero = np.nonzero(mask == 0)[0]
    assert (got["dhv"][zero] == 0).all()
    if rows is None:
        check_grad(got["dhv"], ref["dhv"], zero, "dhidden_value")
    else:
        check_grad(got["dhv"][rows], ref["dhv"][rows], None, "dhidden_value rows")


def check_loss(got, ref, lp, lro, adv, mask, N, propagated_floor=False):
    """Loss values against the oracle: relative 1e-3, guarded against cancellation by
    (1/N) sum |terms|. With `propagated_floor` (only where log pi is exactly 0, so
    that the reference loss and its scale are 0) the bar is at least 4x the loss
    change that the measured log-prob differences account for."""
    rho = np.exp(lp - lro)
    used = (ref["flags"] == 1)
    n = max(N, 1)
    scale0 = np.abs(rho * adv * lp)[used].sum() / n
    scale1 = np.abs(rho * adv)[used].sum() / n
    # d(rho logp)/dlogp = rho (1 + logp) and d(rho)/dlogp = rho: the loss change that
    # the measured log-prob differences alone account for
    dlp = np.abs(np.asarray(got["logp"], dtype=np.float64) - lp)
    prop0 = (np.abs(rho * adv * (1.0 + lp)) * dlp)[used].sum() / n
    prop1 = (np.abs(rho * adv) * dlp)[used].sum() / n
    for k, sc, prop in ((0, scale0, prop0), (1, scale1, prop1)):
        tol = TOL_LOSS * max(abs(ref["loss"][k]), sc, 1e-300)
        if propagated_floor:
            tol = max(tol, 4.0 * prop)
        assert abs(got["loss"][k] - ref["loss"][k]) <= tol, (k, got["loss"][k], ref["loss"][k], tol)


def check_grad(got, ref, rows_zero=None, name="grad"):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    nr = np.linalg.norm(ref)
    if nr == 0:
        assert np.abs(got).max() == 0, name
        return
    assert np.linalg.norm(got - ref) <= TOL_GRAD * nr, (name, np.linalg.norm(got - ref) / nr)
    rn = np.linalg.norm(ref, axis=1)
    big = rn > 1e-3 * rn.max()
    rel = np.linalg.norm(got - ref, axis=1)[big] / rn[big]
    assert rel.max() <= TOL_GRAD, (name, rel.max())
    if rows_zero is not None:
        assert (got[rows_zero] == 0).all(), name


def compare_all(got, ref, batch, backward=True):
    m = batch.mask == 1
    assert np.abs(got["logp"][m] - ref["logp"][m]).max() <= TOL_LOGP
    assert np.abs(got["lse"][m] - ref["lse"][m]).max() <= TOL_LOGP
    assert (got["logp"][~m] == 0).all() and (got["lse"][~m] == 0).all()
    assert int(got["n"][0]) == ref["n"]
    scale = np.maximum(1.0, np.abs(ref["adv"]))
    assert (np.abs(got["adv"] - ref["adv"]) <= TOL_ADV * scale).all()
    scale = np.maximum(1.0, np.abs(ref["ret"]))
    assert (np.abs(got["ret"] - ref["ret"]) <= TOL_ADV * scale).all()
    assert np.array_equal(got["flags"], ref["flags"])
    assert np.array_equal(got["counts"], ref["counts"])
    check_loss(got, ref, ref["logp"], ref["lro"], ref["adv"], batch.mask, ref["n"])
    assert (np.abs(got["g"] - ref["g"]) <= TOL_G * np.abs(ref["g"]) + 1e-12).all()
    assert (got["g"][ref["flags"] != 1] == 0).all()
    if backward:
        zero_rows = np.nonzero(ref["g"] == 0)[0]
        check_grad(got["dh"], ref["dh"], zero_rows, "dhidden")
        check_grad(got["dw"], ref["dw"], None, "dw_head")
    if "lv" in ref:
        check_value(got, ref, batch.mask)
