"""A whole step of the pass captured in a HIP graph and replayed.

The library allocates nothing and never synchronises, so one step (critic,
scan, head forward, loss, backward) on preallocated buffers can be captured.
Each replay, with unrelated eager work in between, must reproduce the eager
step bit for bit: every kernel is deterministic. The accumulating outputs are
zeroed inside the graph by fill kernels.
"""
import numpy as np
import pytest
import torch

import paper_2607_07508_amd as sao
from paper_2607_07508_amd import binding as B
from synth import generate, small_config
from synth.device import to_device
from tests.gpu_common import oracle_pass, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    sao.lib()


def test_captured_step_replays_match_eager():
    cfg = small_config("graph", 51, B=4, T=1500, H=192, V=3000, value_head=True)
    say(f"case {cfg.name}: T={cfg.T} H={cfg.H} V={cfg.V}")
    b = generate(cfg)
    ref = oracle_pass(b, 1.0, 1.0, 1.5, backward=False)
    db = to_device(b, ref["logp"])
    L = sao.lib()
    T, H, V = b.T, cfg.H, cfg.V
    dev = db.hidden.device
    f32 = dict(dtype=torch.float32, device=dev)
    out = dict(v=torch.empty(T, **f32), adv=torch.empty(T, **f32), ret=torch.empty(T, **f32),
               logp=torch.empty(T, **f32), lse=torch.empty(T, **f32), g=torch.empty(T, **f32),
               flags=torch.empty(T, dtype=torch.uint8, device=dev), n=torch.zeros(1, dtype=torch.int64, device=dev),
               loss=torch.zeros(2, dtype=torch.float64, device=dev),
               counts=torch.zeros(5, dtype=torch.int64, device=dev),
               dh=torch.empty((T, H), dtype=db.hidden.dtype, device=dev), dw=torch.zeros((V, H), **f32),
               lv=torch.zeros(1, dtype=torch.float64, device=dev),
               dhv=torch.empty((T, H), dtype=db.hidden.dtype, device=dev), dwv=torch.zeros(H, **f32))
    dt = B.SAO_BF16
    ws_bytes = max(B.workspace_size(op, T, H, V, dt) for op in
                   (B.OP_LOGPROB, B.OP_BACKWARD, B.OP_LOSS, B.OP_ADVANTAGE, B.OP_VALUE))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    p = lambda t: t.data_ptr()  # noqa: E731
    o = out

    def step():
        st = torch.cuda.current_stream().cuda_stream
        for k in ("loss", "counts", "dw", "lv", "dwv"):
            o[k].zero_()
        B._check(L.sao_value_forward(p(db.hidden), H, p(db.w_value), T, H, dt, p(o["v"]), None, 0, st))
        B._check(L.sao_advantage(p(o["v"]), p(db.rewards), p(db.mask), p(db.cu_seqlens), cfg.B, T, 1.0, 1.0, 1.5,
                                 p(o["adv"]), p(o["ret"]), p(o["n"]), None, p(ws), ws_bytes, st))
        B._check(L.sao_value_loss(p(db.hidden), H, p(db.w_value), p(o["v"]), p(o["ret"]), p(db.mask), T, H,
                                  p(o["n"]), dt, p(o["lv"]), p(o["dhv"]), p(o["dwv"]), p(ws), ws_bytes, st))
        B._check(L.sao_token_logprob(p(db.hidden), H, p(db.w_head), H, p(db.target), p(db.mask), T, H, V, dt,
                                     p(o["logp"]), p(o["lse"]), None, p(ws), ws_bytes, st))
        B._check(L.sao_clipped_loss(p(o["logp"]), p(db.logp_rollout), p(o["adv"]), p(db.mask), T, cfg.eps_low,
                                    cfg.eps_high, p(o["n"]), p(o["loss"]), p(o["g"]), p(o["flags"]), p(o["counts"]),
                                    p(ws), ws_bytes, st))
        B._check(L.sao_loss_backward(p(db.hidden), H, p(db.w_head), H, p(db.target), p(o["lse"]), p(o["g"]), T, H,
                                     V, dt, p(o["dh"]), p(o["dw"]), p(ws), ws_bytes, st))

    def snapshot():
        torch.cuda.synchronize()
        return {k: v.clone() for k, v in out.items()}

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm up on a side stream, as graph capture wants
        step()
    torch.cuda.current_stream().wait_stream(side)
    step()
    eager = snapshot()
    assert int(eager["counts"][0]) == int(b.mask.sum()) and np.array_equal(eager["counts"].cpu().numpy(),
                                                                          ref["counts"])
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for i in range(3):
        for v in out.values():       # scribble over the outputs between replays
            v.fill_(7)
        junk = torch.randn(1 << 20, device=dev).sum()   # unrelated eager work
        graph.replay()
        got = snapshot()
        del junk
        for k in out:
            assert torch.equal(got[k], eager[k]), (i, k)
        say(f"replay {i}: identical to the eager step")


def test_captured_comparison_and_baselines_replay_match_eager():
    """The clipped surrogate, explained variance, step-level GAE and both critic-free
    baselines, captured in one graph. The running-mean state is restored eagerly before
    each replay, so every replay starts from the same history."""
    cfg = small_config("graph2", 52, B=8, T=4000, H=8, V=8)
    say(f"case {cfg.name}: T={cfg.T} B={cfg.B}")
    b = generate(cfg, with_head=False)
    from synth import comparison_logprobs
    lp, lold, lb = comparison_logprobs(cfg, b.T)
    dev = torch.device("cuda")
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)  # noqa: E731
    values, rewards, mask, cu = t(b.values), t(b.rewards), t(b.mask), t(b.cu_seqlens)
    lp_d, lold_d, lb_d = t(lp), t(lold), t(lb)
    T, Bn = b.T, cfg.B
    L = sao.lib()
    f32 = dict(dtype=torch.float32, device=dev)
    f64 = dict(dtype=torch.float64, device=dev)
    out = dict(adv=torch.empty(T, **f32), ret=torch.empty(T, **f32), n=torch.zeros(1, dtype=torch.int64, device=dev),
               g=torch.empty(T, **f32), flags=torch.empty(T, dtype=torch.uint8, device=dev),
               loss=torch.zeros(1, **f64), counts=torch.zeros(5, dtype=torch.int64, device=dev),
               mom=torch.zeros(5, **f64), ev=torch.zeros(1, **f64),
               sadv=torch.empty(T, **f32), sret=torch.empty(T, **f32), last=torch.empty(T, dtype=torch.uint8, device=dev),
               gadv=torch.empty(T, **f32), gR=torch.empty(Bn, **f64), gA=torch.empty(Bn, **f64),
               radv=torch.empty(T, **f32), rR=torch.empty(Bn, **f64), rA=torch.empty(Bn, **f64))
    hist0 = torch.rand((2, 4), **f64)
    seen0 = torch.tensor([3, 9], dtype=torch.int64, device=dev)
    hist, seen = hist0.clone(), seen0.clone()
    keys = t((np.arange(Bn) % 2).astype(np.int32))
    ws_bytes = max(B.workspace_size(op, T, 1, 1, B.SAO_F32) for op in
                   (B.OP_ADVANTAGE, B.OP_PPO_LOSS, B.OP_EXPLAINED_VARIANCE, B.OP_STEP_ADVANTAGE,
                    B.OP_GROUP_ADVANTAGE, B.OP_RUNNING_MEAN_ADVANTAGE))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    p = lambda x: x.data_ptr()  # noqa: E731
    o = out

    def step():
        st = torch.cuda.current_stream().cuda_stream
        for k in ("loss", "counts", "mom"):
            o[k].zero_()
        B._check(L.sao_advantage(p(values), p(rewards), p(mask), p(cu), Bn, T, 1.0, 1.0, 1.5, p(o["adv"]),
                                 p(o["ret"]), p(o["n"]), None, p(ws), ws_bytes, st))
        B._check(L.sao_ppo_loss(p(lp_d), p(lold_d), p(lb_d), p(o["adv"]), p(mask), T, 0.2, 0.28, p(o["n"]),
                                p(o["loss"]), p(o["g"]), p(o["flags"]), p(o["counts"]), p(ws), ws_bytes, st))
        B._check(L.sao_explained_variance(p(values), p(o["ret"]), p(mask), T, p(o["mom"]), p(o["ev"]), p(ws),
                                          ws_bytes, st))
        B._check(L.sao_step_advantage(p(values), p(rewards), p(mask), p(cu), Bn, T, 1.0, 1.0, 1.5, B.STEP_LAST,
                                      p(o["sadv"]), p(o["sret"]), p(o["last"]), None, None, p(ws), ws_bytes, st))
        B._check(L.sao_group_advantage(p(rewards), p(mask), p(cu), Bn, T, 4, 1e-6, p(o["gadv"]), p(o["gR"]),
                                       p(o["gA"]), None, None, p(ws), ws_bytes, st))
        B._check(L.sao_running_mean_advantage(p(rewards), p(mask), p(cu), Bn, T, p(keys), 2, 4, p(hist), p(seen),
                                              p(o["radv"]), p(o["rR"]), p(o["rA"]), None, None, p(ws), ws_bytes, st))

    def snapshot():
        torch.cuda.synchronize()
        return {k: v.clone() for k, v in list(out.items()) + [("hist", hist), ("seen", seen)]}

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    hist.copy_(hist0)
    seen.copy_(seen0)
    step()
    eager = snapshot()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for i in range(3):
        for v in out.values():
            v.fill_(7)
        hist.copy_(hist0)
        seen.copy_(seen0)
        junk = torch.randn(1 << 20, device=dev).sum()
        graph.replay()
        got = snapshot()
        del junk
        for k in eager:
            assert torch.equal(got[k], eager[k]), (i, k)
        say(f"replay {i}: identical to the eager calls")
