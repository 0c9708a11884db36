#!/usr/bin/env python3
"""Throughput of the SAO per-token loss pass on one MI355X.

One step is the whole hot path over one synthetic batch: skip-observation GAE
(sao_advantage), LM-head log-probs (sao_token_logprob), the DIS loss
(sao_clipped_loss) and the backward into hidden states and W_head
(sao_loss_backward), with the zeroing of the accumulated outputs. Inputs are
resident in HBM before the timed region.

Default workload (c2): 16 single rollouts, T = 65,536 tokens, H = 2048,
V = 151,936, bf16 hidden/W_head, forward + backward, drift noise sigma 0.2.
--workload c1 / c3 / c4 run the forward-only, the long-horizon chunked and the
large-head-with-critic workloads the same way (reported, not the headline).

Prints one JSON line (rank 0, one GPU): tokens/s, the roofline figure of the
head-forward MFMA kernel (timed live with HIP events around its launches) and
the fp64 oracle timed on this host's cores over a bounded sample of the batch.
"""
from __future__ import annotations

import argparse
import contextlib
import json
import os
import sys
import time

import numpy as np
from typing import Optional

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tokens/s SAO logprob+clipped-loss fwd+bwd (H2048,V152k); % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 MFMA, TFLOP/s
PEAK_HBM_GBS = 8000.0              # MI355X HBM3E, GB/s
WORKLOAD_TEXT = {
    "c1": "16 single rollouts, T=65536, H=2048, V=151936, bf16, forward only (log-probs, scan, loss), "
          "~30% observation tokens, drift sigma 0.1, eps 0.2/0.2, gamma 1, alpha 1.5",
    "c2": "16 single rollouts, T=65536, H=2048, V=151936, bf16, fwd+bwd, ~30% observation tokens, "
          "drift sigma 0.2, eps 0.2/0.2, gamma 1, alpha 1.5",
    "c3": "8 long-horizon rollouts (Pareto lengths, cap 65536), T=262144, H=2048, V=151936, bf16, fwd+bwd in "
          "32 chunks of 8192 tokens with the whole-batch scan and N, ~50% observation tokens, eps 0.2/0.2",
    "c4": "64 single rollouts, T=32768, H=6144, V=151552, bf16, fwd+bwd plus the critic head (values from "
          "h.w_v, squared-error loss), ~25% observation tokens, eps 0.2/0.28",
}


KERNEL_SOURCES = ["paper_2607_07508_amd/csrc/gemm.hpp", "paper_2607_07508_amd/csrc/head.hip",
                  "paper_2607_07508_amd/csrc/common.hpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "head_fwd_c2_traffic.json")


def kernel_source_sha() -> str:
    """Hash of the head kernels' code: their sources with comments and whitespace
    removed, so that an edit of a comment does not mark the counters stale."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per head-forward launch from the committed counter runs, or None
    when the kernel sources changed since those counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    if d.get("source_sha") != kernel_source_sha():
        return None
    return d.get("bytes_per_launch")


def copy_calibration(nbytes: int = 1 << 30):
    """A plain device copy of known size, for scaling the FETCH_SIZE/WRITE_SIZE counters."""
    import torch
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "launches": 3}), flush=True)


def backward_vocab_block(T: int, V: int, H: int, esize: int = 2) -> int:
    """Vocabulary rows per block of sao_loss_backward for T token rows (the rule of
    csrc/layout.hpp: a 32,768-row target, doubled up to 65,536 while the dz product
    has fewer than 8192 tiles, then V cut into that many near-equal blocks, each
    rounded to a whole number of rounds of its dW tiles on 256 CUs: up where the
    block's rows of W then fit the 256 MB memory-side cache, else down)."""
    import math
    tiles_t = -(-T // 256)
    vc = 32768
    while vc < 65536 and tiles_t * (vc // 256) < 8192:
        vc *= 2
    blocks = -(-V // vc)
    tiles = -(-(-(-V // blocks)) // 256)
    align = 256 // math.gcd(256, -(-H // 256))
    rounded = -(-tiles // align) * align
    if blocks > 1 and rounded <= vc // 256 and rounded * 256 * H * esize <= 256 << 20:
        tiles = rounded
    elif blocks > 1 and tiles >= align:
        tiles = tiles // align * align
    return tiles * 256


def wall_clock_khz() -> Optional[int]:
    """The device's constant wall-clock rate (hipDeviceAttributeWallClockRate), in kHz."""
    import ctypes
    try:
        hip = ctypes.CDLL("libamdhip64.so")
        v = ctypes.c_int(0)
        if hip.hipDeviceGetAttribute(ctypes.byref(v), 10017, 0) != 0:  # hipDeviceAttributeWallClockRate
            return None
        return int(v.value) or None
    except OSError:
        return None


def kernel_timeline(step, torch, dev, B, kernel=None):
    """One more step (after the timed ones) with a head kernel's own per-workgroup
    records on (default the head forward; the step's last launch of it stays
    recorded, for the backward kernels the first vocabulary block's). Returns the
    records as a numpy int64 [n, 8] array of the workgroups that ran a tile, and
    the wall-clock rate in kHz."""
    rec = torch.zeros((1 << 18, 8), dtype=torch.int64, device=dev)
    try:
        B.clock_samples(rec, B.KERNEL_HEAD_FORWARD if kernel is None else kernel)
        step()
        torch.cuda.synchronize()
    finally:
        B.clock_samples(None)
    r = rec.cpu().numpy()
    return r[(r[:, 2] > r[:, 1]) & (r[:, 7] >= 0)], wall_clock_khz()


def forward_clock(step, torch, dev, B) -> dict:
    """The shader clock the head-forward kernel ran at: s_memtime cycles over
    s_memrealtime time, summed over its workgroups."""
    r, khz = kernel_timeline(step, torch, dev, B)
    if not khz or r.shape[0] == 0:
        return {"forward_clock_mhz": None, "clock_note": "wall-clock rate or records unavailable"}
    cycles, ticks = float((r[:, 6] - r[:, 3]).sum()), float((r[:, 2] - r[:, 1]).sum())
    return {"forward_clock_mhz": cycles / (ticks / (khz * 1e3)) / 1e6,
            "clock_note": "shader clock of k_head_fwd's workgroups over one step (s_memtime cycles over "
                          "s_memrealtime time, last forward launch of the step)"}


def timeline_summary(r, khz, k=None) -> dict:
    """Where a head kernel's tile time goes: per-tile prologue, K loop and epilogue
    cycles, and per CU the wall-clock gaps between one workgroup's end and the next
    one's start, in cycles at the measured clock; the range of the CUs' busy
    fractions and of the tiles per shader engine (XCC and SE from the hardware
    ids). With the contraction length k,
    also the MFMA cycles a tile needs (256 x 256 x k x 2 flop at 4 SIMDs x 1024
    bf16 flop per cycle) and the K loop's MFMA efficiency."""
    clk = (r[:, 6] - r[:, 3]).sum() / ((r[:, 2] - r[:, 1]).sum() / (khz * 1e3))
    pro, loop, epi = r[:, 4] - r[:, 3], r[:, 5] - r[:, 4], r[:, 6] - r[:, 5]
    hw = r[:, 0]
    cu = ((hw >> 32) << 16) | (((hw >> 13) & 7) << 8) | (((hw >> 12) & 1) << 4) | ((hw >> 8) & 15)
    gaps, per_cu = [], {}
    for c in np.unique(cu):
        sel = np.nonzero(cu == c)[0]
        o = sel[np.argsort(r[sel, 1])]
        g = (r[o[1:], 1] - r[o[:-1], 2]) / (khz * 1e3) * clk
        gaps.append(g)
        per_cu[int(c)] = int(o.size)
    g = np.concatenate(gaps) if gaps else np.zeros(0)
    span = (r[:, 2].max() - r[:, 1].min()) / (khz * 1e3)
    busy = ((r[:, 2] - r[:, 1]).sum() / (khz * 1e3)) / (len(per_cu) * span)
    # per CU, the fraction of the span it held a tile; per shader engine (XCC, SE), its tiles
    held = [((r[cu == c, 2] - r[cu == c, 1]).sum() / (khz * 1e3)) / span for c in per_cu]
    se = (hw >> 32) * 8 + ((hw >> 13) & 7)
    per_se = np.unique(se, return_counts=True)[1]
    mfma = 256 * 256 * 2 * k / 4096 if k else None
    return {"clock_mhz": clk / 1e6, "tiles": int(r.shape[0]), "cus": len(per_cu),
            "k": k, "mfma_cycles_per_tile": mfma,
            "k_loop_mfma_efficiency": float(mfma / loop.mean()) if mfma else None,
            "tiles_per_cu": [int(min(per_cu.values())), int(max(per_cu.values()))],
            "cycles_per_tile": {"prologue": float(pro.mean()), "k_loop": float(loop.mean()),
                                "epilogue": float(epi.mean()), "total": float((pro + loop + epi).mean())},
            "gap_cycles_between_tiles": {"median": float(np.median(g)) if g.size else None,
                                         "mean": float(g.mean()) if g.size else None},
            "cu_busy_fraction": float(busy), "cu_busy_range": [float(min(held)), float(max(held))],
            "tiles_per_shader_engine": [int(per_se.min()), int(per_se.max())],
            "launch_span_ms": float(span * 1e3)}


def vendor_gemm(db, t_act: int, t_grad: int, vc: int, torch, reps: int = 3):
    """torch.matmul (hipBLASLt) in bf16 at the four head-contraction shapes the
    library runs on MFMA, for context only (run, never inspected):
      forward       (T_act x H) . (H x V)       on the batch's hidden rows and W_head
      dz recompute  (T_grad x H) . (H x Vb)     one backward vocabulary block of W_head
      dH            (T_grad x Vb) . (Vb x H)
      dW            (Vb x T_grad) . (T_grad x H)
    Vb is the library's full backward block. Every operand is contiguous (no
    transposed views); the dz operands are random, scaled like small gradients.
    The library kernels' own times come from the kernel trace of the same run."""
    H = db.hidden.shape[1]
    w = db.w_head
    gen = torch.Generator(device=db.hidden.device).manual_seed(7)
    hg = db.hidden[:t_grad].contiguous()
    dz = (torch.randn(t_grad, vc, generator=gen, device=db.hidden.device) * 1e-4).to(torch.bfloat16)
    shapes = {
        "forward": (lambda: db.hidden[:t_act].contiguous(), lambda: w.t().contiguous(), t_act, w.shape[0], H),
        "dz_recompute": (lambda: hg, lambda: w[:vc].t().contiguous(), t_grad, vc, H),
        "dH": (lambda: dz, lambda: w[:vc].contiguous(), t_grad, H, vc),
        "dW": (lambda: dz.t().contiguous(), lambda: hg, vc, H, t_grad),
    }
    out = {}
    for name, (fa, fb, M, N, K) in shapes.items():
        a, b = fa(), fb()
        c = torch.matmul(a, b)
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record()
        for _ in range(reps):
            torch.matmul(a, b, out=c)
        ev1.record()
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1) / reps
        flops = 2.0 * M * N * K
        out[name] = {"op": f"torch.matmul bf16 ({M} x {K}) . ({K} x {N})", "M": M, "N": N, "K": K, "ms": ms,
                     "TFLOP/s": flops / ms / 1e9, "frac": flops / ms / 1e9 / PEAK_BF16_TFLOPS}
        del a, b, c
        torch.cuda.empty_cache()
    del hg, dz
    torch.cuda.empty_cache()
    return out


def mfma_ceiling(blocks: int = 2048, iters: int = 20000, reps: int = 3):
    """What the bf16 MFMA pipe delivers with nothing else to issue: the probe library's
    loop of 16 v_mfma_f32_32x32x16_bf16 per round on 256 accumulators, one wave per
    SIMD (the head kernels' arrangement), for random, constant and refreshed-random
    operands; then the same MFMAs fed from LDS the way the tile engine feeds them,
    without and with its global->LDS copies and per-slab barrier, and with both
    operands MN-major through the transposing LDS read (as the backward's dW
    product reads them), without and with the copies. With the clock the
    workgroups ran at. One JSON line per mode."""
    import ctypes
    import torch
    from paper_2607_07508_amd import build as bld
    if not torch.cuda.is_available():
        print("the probe needs a HIP device", file=sys.stderr)
        sys.exit(1)
    lib = ctypes.CDLL(bld.PROBE_LIB)
    fn = lib.sao_probe_mfma
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                   ctypes.c_void_p]
    # 2 MB of random bf16 bit patterns for mode 4's copies to read
    gen = torch.Generator(device="cuda").manual_seed(3)
    src = (torch.randn((1 << 20,), generator=gen, device="cuda")).to(torch.bfloat16)
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    clk = torch.zeros((blocks, 3), dtype=torch.int64, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    khz = wall_clock_khz()
    flops = 2.0 * 32 * 32 * 16 * 16 * 4 * blocks * iters
    modes = ((0, "random operands"), (1, "constant operands"), (2, "random operands refreshed per round"),
             (3, "random operands read from LDS as the tile engine reads them"),
             (4, "LDS reads plus the engine's global->LDS copies and a barrier per slab"),
             (5, "MN-major operands read from LDS through the transposing read, as dW reads them"),
             (6, "transposing LDS reads plus the engine's copies and a barrier per slab"))
    for mode, name in modes:
        if fn(blocks, iters, mode, src.data_ptr(), out.data_ptr(), clk.data_ptr(), st) != 0:
            raise RuntimeError("probe launch failed")
        torch.cuda.synchronize()
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn(blocks, iters, mode, src.data_ptr(), out.data_ptr(), clk.data_ptr(), st)
        z.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(z) / reps
        r = clk.cpu().numpy()
        cyc, ticks = float(r[:, 0].sum()), float((r[:, 2] - r[:, 1]).sum())
        mhz = cyc / (ticks / (khz * 1e3)) / 1e6 if khz and ticks else None
        tf = flops / ms / 1e9
        print(json.dumps({"mode": "mfma_ceiling", "operands": name, "ms": ms, "TFLOP/s": tf,
                          "frac": tf / PEAK_BF16_TFLOPS, "clock_mhz": mhz,
                          "frac_at_clock": (tf / (PEAK_BF16_TFLOPS * mhz / 2400.0)) if mhz else None,
                          "blocks": blocks, "iters": iters}), flush=True)


def epilogue_sweep(exps=(20, 22, 24, 26), reps=20):
    """Achieved HBM bandwidth of the scan (sao_advantage), the loss epilogue
    (sao_clipped_loss), the decoupled clipped surrogate (sao_ppo_loss with
    logp_behav) and the explained variance (sao_explained_variance) at T = 2^e
    tokens, B = T/4096 trajectories, c2's span mix. Algorithmic bytes per token:
    17 for the scan (values, rewards, mask in; adv, ret out), 18 for the loss
    (logp, logp_rollout, adv, mask in; g, flags out), 22 for the surrogate
    (logp, logp_old, logp_behav, adv, mask in; g, flags out), 9 for the
    explained variance (values, ret, mask in), and for the step-level GAE
    (sao_step_advantage, step averages) 14 per token plus 4 per loss-mask token
    (mask and rewards in, adv, ret and last out; values only on the steps),
    and 9 for the critic-free baselines (sao_group_advantage with groups of 8,
    sao_running_mean_advantage with one 128-reward window: rewards and mask in,
    adv out). One JSON line per size."""
    import torch
    import paper_2607_07508_amd as sao
    from paper_2607_07508_amd import binding as B
    from synth import generate, small_config
    from synth.device import to_device
    if not torch.cuda.is_available():
        print("the sweep needs a HIP device", file=sys.stderr)
        sys.exit(1)
    # Reference: a plain device copy (1 GiB read + 1 GiB written) on the same box.
    src = torch.empty(1 << 28, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    z.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(z) / reps
    print(json.dumps({"mode": "copy_reference", "bytes": 2 << 30, "ms": ms, "GB/s": (2 << 30) / ms / 1e6,
                      "frac_hbm": (2 << 30) / ms / 1e6 / PEAK_HBM_GBS}), flush=True)
    del src, dst
    torch.cuda.empty_cache()
    for e in exps:
        T = 1 << e
        cfg = small_config(f"sweep{e}", 2000 + e, B=T // 4096, T=T, H=8, V=16,
                           length=("lognormal", 4096, 0.5, 16384), act_span=(800, 2400), obs_span=(64, 2048))
        log(f"sweep T=2^{e}: generating")
        b = generate(cfg, with_head=False)
        db = to_device(b)
        g = torch.Generator(device="cpu").manual_seed(e)
        logp = (-torch.rand(T, generator=g) * 4.0).to("cuda")
        lro = logp + torch.from_numpy(b.xi).float().to("cuda")
        lbh = lro + 0.05 * torch.randn(T, generator=g).to("cuda")
        L = sao.lib()
        f32 = dict(dtype=torch.float32, device="cuda")
        adv, ret, g_out = torch.empty(T, **f32), torch.empty(T, **f32), torch.empty(T, **f32)
        flags = torch.empty(T, dtype=torch.uint8, device="cuda")
        n = torch.zeros(1, dtype=torch.int64, device="cuda")
        loss = torch.zeros(2, dtype=torch.float64, device="cuda")
        counts = torch.zeros(5, dtype=torch.int64, device="cuda")
        moments = torch.zeros(5, dtype=torch.float64, device="cuda")
        ev = torch.zeros(1, dtype=torch.float64, device="cuda")
        ws_bytes = max(B.workspace_size(op, T, 1, 1, B.SAO_F32)
                       for op in (B.OP_ADVANTAGE, B.OP_LOSS, B.OP_PPO_LOSS, B.OP_EXPLAINED_VARIANCE,
                                  B.OP_GROUP_ADVANTAGE, B.OP_RUNNING_MEAN_ADVANTAGE))
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        st = torch.cuda.current_stream().cuda_stream
        p = lambda t: t.data_ptr()  # noqa: E731

        def scan():
            B._check(L.sao_advantage(p(db.values), p(db.rewards), p(db.mask), p(db.cu_seqlens), cfg.B, T, 1.0, 1.0,
                                     1.5, p(adv), p(ret), p(n), None, p(ws), ws_bytes, st))

        def epilogue():
            B._check(L.sao_clipped_loss(p(logp), p(lro), p(adv), p(db.mask), T, 0.2, 0.2, p(n), p(loss), p(g_out),
                                        p(flags), p(counts), p(ws), ws_bytes, st))
        def surrogate():
            B._check(L.sao_ppo_loss(p(logp), p(lro), p(lbh), p(adv), p(db.mask), T, 0.2, 0.28, p(n), p(loss),
                                    p(g_out), p(flags), p(counts), p(ws), ws_bytes, st))

        last = torch.empty(T, dtype=torch.uint8, device="cuda")
        step_ws = torch.empty(B.workspace_size(B.OP_STEP_ADVANTAGE, T, 1, 1, B.SAO_F32), dtype=torch.uint8,
                              device="cuda")

        def step_gae():
            B._check(L.sao_step_advantage(p(db.values), p(db.rewards), p(db.mask), p(db.cu_seqlens), cfg.B, T, 1.0,
                                          1.0, 1.5, B.STEP_AVERAGE, p(g_out), p(ret), p(last), p(n), None,
                                          p(step_ws), step_ws.numel(), st))

        traj_r = torch.empty(cfg.B, dtype=torch.float64, device="cuda")
        traj_a = torch.empty(cfg.B, dtype=torch.float64, device="cuda")
        hist, seen = torch.zeros(128, dtype=torch.float64, device="cuda"), torch.zeros(1, dtype=torch.int64,
                                                                                        device="cuda")

        def grpo():
            B._check(L.sao_group_advantage(p(db.rewards), p(db.mask), p(db.cu_seqlens), cfg.B, T, 8, 1e-6, p(g_out),
                                           p(traj_r), p(traj_a), p(n), None, p(ws), ws_bytes, st))

        def running_mean():
            B._check(L.sao_running_mean_advantage(p(db.rewards), p(db.mask), p(db.cu_seqlens), cfg.B, T, None, 1, 128,
                                                  p(hist), p(seen), p(g_out), p(traj_r), p(traj_a), p(n), None,
                                                  p(ws), ws_bytes, st))

        def explained():
            B._check(L.sao_explained_variance(p(db.values), p(ret), p(db.mask), T, p(moments), p(ev), p(ws), ws_bytes,
                                              st))
        out = {}
        for name, fn, nbytes in (("advantage", scan, 17 * T), ("clipped_loss", epilogue, 18 * T),
                                 ("ppo_loss", surrogate, 22 * T), ("explained_variance", explained, 9 * T),
                                 ("step_advantage", step_gae, 14 * T + 4 * int(b.mask.sum())),
                                 ("group_advantage", grpo, 9 * T), ("running_mean_advantage", running_mean, 9 * T)):
            for _ in range(3):
                fn()
            torch.cuda.synchronize()
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                fn()
            z.record()
            torch.cuda.synchronize()
            ms = a.elapsed_time(z) / reps
            out[name] = {"ms": ms, "GB/s": nbytes / ms / 1e6, "frac_hbm": nbytes / ms / 1e6 / PEAK_HBM_GBS,
                         "bytes": nbytes}
        print(json.dumps({"mode": "epilogue_sweep", "T": T, "B": cfg.B, **out}), flush=True)
        del db, b, logp, lro, lbh, adv, ret, g_out, flags, ws, last, step_ws, traj_r, traj_a, hist, seen
        torch.cuda.empty_cache()


def breakdown(step, T, H, V, esz, t_act, t_grad, torch, repeats=3):
    """`repeats` more steps, after the timed ones, with each library call bracketed
    by events on the launch stream: per-call device time (summed over chunks, the
    median over the repeats) and its rate against the roofline that bounds it.
    Not part of `value`."""
    runs = []
    for _ in range(repeats):
        spans = {}

        @contextlib.contextmanager
        def span(name):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            yield
            b.record()
            spans.setdefault(name, []).append((a, b))

        step(span=span)
        torch.cuda.synchronize()
        runs.append({k: sum(a.elapsed_time(b) for a, b in v) for k, v in spans.items()})
    ms = {k: float(np.median([r[k] for r in runs])) for k in runs[0]}
    # bytes: the per-token arrays, and for the critic the hidden rows read (and dH_v written)
    hbm = {"advantage": 17.0 * T, "clipped_loss": 18.0 * T, "value_forward": esz * T * H + 4.0 * T,
           "value_loss": 2.0 * esz * T * H + 13.0 * T}
    flops = {"token_logprob": 2.0 * t_act * V * H,
             "loss_backward": 6.0 * t_grad * V * H}   # logits recomputed, dH, dW
    out = {}
    for k, t in ms.items():
        row = {"ms": t}
        if k in flops:
            row.update({"TFLOP/s": flops[k] / (t * 1e-3) / 1e12, "frac": flops[k] / (t * 1e-3) / 1e12 /
                        PEAK_BF16_TFLOPS, "bound": "mfma"})
        elif k in hbm:
            row.update({"GB/s": hbm[k] / (t * 1e-3) / 1e9, "frac": hbm[k] / (t * 1e-3) / 1e9 / PEAK_HBM_GBS,
                        "bound": "hbm"})
        out[k] = row
    return out


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(batch, ref_logp, rows: int, seed: int = 0):
    """The oracle on a bounded sample: `rows` loss-mask tokens (default: a quarter of
    them) through the head pass (forward, and backward for those with g != 0), plus
    the whole-batch scan and loss; scaled to the whole batch by the share of
    loss-mask tokens sampled."""
    import oracle
    from synth import rollout_logprobs
    try:
        from threadpoolctl import threadpool_info
        blas = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas = None
    cores = len(os.sched_getaffinity(0))
    cfg = batch.cfg
    act = np.nonzero(batch.mask)[0]
    rng = np.random.default_rng(seed)
    n = act.size // 4 if rows <= 0 else min(rows, act.size)
    sample = np.sort(rng.choice(act, size=n, replace=False))
    t0 = time.perf_counter()
    w64 = batch.w_head.astype(np.float64)
    adv, ret, N = oracle.advantage(batch.values, batch.rewards, batch.mask, batch.cu_seqlens, cfg.gamma,
                                   cfg.lam, cfg.alpha)
    t_scan = time.perf_counter() - t0
    t1 = time.perf_counter()
    lp, lse = oracle.token_logprob(batch.hidden, None, batch.target, rows=sample, w64=w64)
    lro = rollout_logprobs(ref_logp, batch.xi)
    sub = np.zeros_like(batch.mask)
    sub[sample] = 1
    _, g, _, _ = oracle.dis_loss(lp, lro, adv, sub, cfg.eps_low, cfg.eps_high, N)
    oracle.loss_backward(batch.hidden, None, batch.target, lse, g, w64=w64)
    t_head = time.perf_counter() - t1
    est = t_scan + t_head * act.size / sample.size
    return {"value": batch.T / est, "unit": "tokens/s", "cores": cores, "blas_threads": blas, "kind": "oracle",
            "sample": f"{sample.size} of {act.size} loss-mask tokens ({sample.size / act.size:.0%}) through the "
                      f"fp64 head forward+backward ({t_head:.1f} s, scaled by {act.size / sample.size:.2f}) plus "
                      f"the whole-batch scan and loss ({t_scan:.1f} s); W_head widening to fp64 excluded; "
                      f"{cores} host cores visible, BLAS on {blas} threads"}



def cpu_baseline_full(names=("c0", "c1", "c2", "c4", "c3"), chunk_rows: int = 8192):
    """The oracle on whole workloads, on the host's cores: the forward over every
    loss-mask row, the scan and loss over the batch, the backward over every row
    with g != 0 where the workload has a backward (not c1), and the critic for c4,
    each timed; the head work goes in chunks
    of rows so that a progress line appears every few tens of seconds. c3 runs
    the head on the rows of its first 8 of 32 token chunks and is scaled by 4
    (labelled as extrapolated). One JSON line per workload."""
    import oracle
    from synth import CONFIGS, generate, rollout_logprobs
    try:
        from threadpoolctl import threadpool_info
        blas = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas = None
    cores = len(os.sched_getaffinity(0))
    for name in names:
        cfg = CONFIGS[name]
        log(f"oracle in full: generating {name}")
        b = generate(cfg)
        T = b.T
        act = np.nonzero(b.mask)[0]
        scale = 1.0
        if name == "c3":
            limit = 8 * cfg.chunk
            head_rows = act[act < limit]
            scale = act.size / head_rows.size
        else:
            head_rows = act
        parts = {}
        w64 = b.w_head.astype(np.float64)
        t = time.perf_counter()
        if cfg.value_head:
            values = oracle.value_forward(b.hidden, b.w_value)
        else:
            values = b.values
        parts["critic_forward"] = time.perf_counter() - t
        t = time.perf_counter()
        adv, ret, N = oracle.advantage(values, b.rewards, b.mask, b.cu_seqlens, cfg.gamma, cfg.lam, cfg.alpha)
        parts["scan"] = time.perf_counter() - t
        t = time.perf_counter()
        lp = np.zeros(T)
        lse = np.zeros(T)
        for s0 in range(0, head_rows.size, chunk_rows):
            r = head_rows[s0:s0 + chunk_rows]
            lp_c, lse_c = oracle.token_logprob(b.hidden, None, b.target, rows=r, w64=w64)
            lp[r], lse[r] = lp_c[r], lse_c[r]
            log(f"oracle in full: {name} forward rows {s0 + r.size} of {head_rows.size}")
        parts["head_forward"] = time.perf_counter() - t
        t = time.perf_counter()
        lro = rollout_logprobs(lp, b.xi)
        sub = np.zeros_like(b.mask)
        sub[head_rows] = 1
        _, g, _, _ = oracle.dis_loss(lp, lro, adv, sub, cfg.eps_low, cfg.eps_high, N)
        parts["loss"] = time.perf_counter() - t
        t = time.perf_counter()
        if cfg.value_head:
            oracle.value_loss(b.hidden, b.w_value, values, ret, b.mask, N)
        parts["critic_loss"] = time.perf_counter() - t
        t = time.perf_counter()
        live = np.nonzero(g)[0] if cfg.backward else np.zeros(0, dtype=np.int64)  # c1 is forward only
        for s0 in range(0, live.size, chunk_rows):
            r = live[s0:s0 + chunk_rows]
            gc = np.zeros_like(g)
            gc[r] = g[r]
            oracle.loss_backward(b.hidden, None, b.target, lse, gc, w64=w64)
            log(f"oracle in full: {name} backward rows {s0 + r.size} of {live.size}")
        parts["head_backward"] = time.perf_counter() - t
        total = (parts["critic_forward"] + parts["scan"] + parts["loss"] + parts["critic_loss"]
                 + (parts["head_forward"] + parts["head_backward"]) * scale)
        print(json.dumps({"mode": "cpu_baseline_full", "workload": name, "T": T, "T_act": int(act.size),
                          "T_grad": int(round(live.size * scale)), "seconds": total, "tokens_per_s": T / total,
                          "parts_seconds": parts, "head_scale": scale, "extrapolated": scale != 1.0,
                          "cores": cores, "blas_threads": blas, "kind": "oracle",
                          "note": ("head forward and backward on the rows of 8 of the 32 token chunks, scaled by "
                                   f"{scale:.2f}; scan, loss and critic on the whole batch") if scale != 1.0
                          else "every loss-mask row; W_head widening to fp64 excluded"}), flush=True)
        del b, w64, lp, lse, g

def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="c2", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--cpu-rows", type=int, default=0,
                    help="loss-mask tokens in the oracle sample (default 0: a quarter of them)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-baseline-full", action="store_true",
                    help="run only the oracle on whole workloads (c0, c1, c2, c4; c3 on 8 of its 32 chunks) on the "
                         "host, one line per workload (minutes)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--vendor-gemm", action="store_true",
                    help="also time torch.matmul (bf16) at the four head shapes (forward; dz, dH and dW of a full "
                         "backward block), as context (allocates the T_act x V output)")
    ap.add_argument("--timeline", action="store_true",
                    help="also record the per-workgroup timelines of the head forward and the backward's three "
                         "products (first vocabulary block), one extra step each")
    ap.add_argument("--mfma-ceiling", action="store_true",
                    help="run only the MFMA probe loops (register operands: random, constant, refreshed; LDS-fed "
                         "without and with the engine's copies; both operands MN-major through the transposing read, "
                         "without and with the copies), one line per mode")
    ap.add_argument("--epilogue-sweep", action="store_true",
                    help="HBM bandwidth of the scan and loss epilogue at T = 2^20 .. 2^26 (one line per size)")
    args = ap.parse_args()
    if args.cpu_baseline_full:
        cpu_baseline_full()
        return
    if args.copy_calibration:
        copy_calibration()
        return
    if args.epilogue_sweep:
        epilogue_sweep()
        return
    if args.mfma_ceiling:
        mfma_ceiling()
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2607_07508_amd as sao
    from paper_2607_07508_amd import binding as B
    from synth import CONFIGS, generate
    from synth.device import to_device
    from tests.golden.make_full_logprobs import load as load_golden

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        sys.exit(1)
    cfg = CONFIGS[args.workload]
    log(f"generating {args.workload}")
    batch = generate(cfg)
    ref_logp, _ = load_golden(args.workload, batch)
    db = to_device(batch, ref_logp)
    L = sao.lib()
    T, H, V = batch.T, cfg.H, cfg.V
    dev = db.hidden.device
    st = torch.cuda.current_stream(dev).cuda_stream
    f32 = dict(dtype=torch.float32, device=dev)

    logp = torch.empty(T, **f32)
    lse = torch.empty(T, **f32)
    adv = torch.empty(T, **f32)
    ret = torch.empty(T, **f32)
    g = torch.empty(T, **f32)
    flags = torch.empty(T, dtype=torch.uint8, device=dev)
    n_tok = torch.zeros(1, dtype=torch.int64, device=dev)
    loss = torch.zeros(2, dtype=torch.float64, device=dev)
    counts = torch.zeros(5, dtype=torch.int64, device=dev)
    dhid = torch.empty((T, H), dtype=db.hidden.dtype, device=dev) if cfg.backward else None
    dw = torch.zeros((V, H), **f32) if cfg.backward else None
    dt = B.SAO_BF16 if cfg.dtype == "bf16" else B.SAO_F32
    esz = db.hidden.element_size()
    chunk = cfg.chunk or T
    chunks = [(s0, min(T, s0 + chunk)) for s0 in range(0, T, chunk)]
    ws_bytes = max(B.workspace_size(B.OP_LOGPROB, chunk, H, V, dt), B.workspace_size(B.OP_BACKWARD, chunk, H, V, dt),
                   B.workspace_size(B.OP_LOSS, T, 1, 1, dt), B.workspace_size(B.OP_ADVANTAGE, T, 1, 1, dt),
                   B.workspace_size(B.OP_VALUE, T, H, 1, dt))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    if cfg.value_head:
        v_out = torch.empty(T, **f32)
        loss_v = torch.zeros(1, dtype=torch.float64, device=dev)
        dhid_v = torch.empty((T, H), dtype=db.hidden.dtype, device=dev)
        dw_v = torch.zeros(H, **f32)
    p = lambda t: t.data_ptr()  # noqa: E731
    fwd_pairs = []   # event pairs bracketing the head-forward launches of the timed steps

    def no_span(name):
        return contextlib.nullcontext()

    def step(timed_pairs=None, span=no_span):
        loss.zero_()
        counts.zero_()
        if cfg.backward:
            dw.zero_()
        values = db.values
        if cfg.value_head:
            loss_v.zero_()
            dw_v.zero_()
            with span("value_forward"):
                B._check(L.sao_value_forward(p(db.hidden), H, p(db.w_value), T, H, dt, p(v_out), None, 0, st))
            values = v_out
        with span("advantage"):
            B._check(L.sao_advantage(p(values), p(db.rewards), p(db.mask), p(db.cu_seqlens), cfg.B, T,
                                     cfg.gamma, cfg.lam, cfg.alpha, p(adv), p(ret), p(n_tok), None, p(ws),
                                     ws_bytes, st))
        if cfg.value_head:
            with span("value_loss"):
                B._check(L.sao_value_loss(p(db.hidden), H, p(db.w_value), p(v_out), p(ret), p(db.mask), T, H,
                                          p(n_tok), dt, p(loss_v), p(dhid_v), p(dw_v), p(ws), ws_bytes, st))
        for i, (s0, e0) in enumerate(chunks):
            n = e0 - s0
            if timed_pairs is not None:
                B.time_kernel(B.KERNEL_HEAD_FORWARD, *timed_pairs[i])
            with span("token_logprob"):
                B._check(L.sao_token_logprob(p(db.hidden) + s0 * H * esz, H, p(db.w_head), H,
                                             p(db.target) + 4 * s0, p(db.mask) + s0, n, H, V, dt, p(logp) + 4 * s0,
                                             p(lse) + 4 * s0, None, p(ws), ws_bytes, st))
            with span("clipped_loss"):
                B._check(L.sao_clipped_loss(p(logp) + 4 * s0, p(db.logp_rollout) + 4 * s0, p(adv) + 4 * s0,
                                            p(db.mask) + s0, n, cfg.eps_low, cfg.eps_high, p(n_tok), p(loss),
                                            p(g) + 4 * s0, p(flags) + s0, p(counts), p(ws), ws_bytes, st))
            if cfg.backward:
                with span("loss_backward"):
                    B._check(L.sao_loss_backward(p(db.hidden) + s0 * H * esz, H, p(db.w_head), H,
                                                 p(db.target) + 4 * s0, p(lse) + 4 * s0, p(g) + 4 * s0, n, H, V,
                                                 dt, p(dhid) + s0 * H * esz, p(dw), p(ws), ws_bytes, st))
        if timed_pairs is not None:
            B.time_kernel(B.KERNEL_NONE, None, None)

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    counts_h = counts.cpu().numpy()
    t_act = int(counts_h[0])
    t_grad = int(counts_h[1])

    fwd_ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in chunks] for _ in range(args.steps)]
    step_ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    for pairs in fwd_ev:       # materialise the event handles
        for a, b in pairs:
            a.record()
            b.record()
    for a in step_ev:
        a.record()
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    step_ev[0].record()
    for i in range(args.steps):
        step(fwd_ev[i])
        step_ev[i + 1].record()
    torch.cuda.synchronize()
    B.time_kernel(B.KERNEL_NONE, None, None)
    per_step = [step_ev[i].elapsed_time(step_ev[i + 1]) for i in range(args.steps)]
    ms = step_ev[0].elapsed_time(step_ev[-1]) / args.steps
    # the forward kernel's time per step (all chunks), and per launch
    fwd_step_ms = float(np.mean([sum(a.elapsed_time(b) for a, b in pairs) for pairs in fwd_ev]))
    fwd_ms = fwd_step_ms / len(chunks)

    fwd_flops = 2.0 * t_act * V * H / len(chunks)   # per launch, averaged over the chunks
    achieved = fwd_flops / (fwd_ms * 1e-3) / 1e12
    algo_flops = (2.0 * t_act + (4.0 * t_grad if cfg.backward else 0.0)) * V * H
    out = {
        "metric": METRIC,
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {WORKLOAD_TEXT[args.workload]}", "T": T, "H": H, "V": V,
                   "B": cfg.B, "T_act": t_act, "T_grad": t_grad, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "mfma", "kernel": "k_head_fwd (sao_token_logprob)", "achieved": achieved,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": measured_traffic() if args.workload == "c2" else None, "launch_ms": fwd_ms,
                     "flops_per_launch": fwd_flops},
        "algorithmic_mfma_frac": algo_flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        "step_ms": {"median": float(np.median(per_step)), "min": float(np.min(per_step)),
                    "max": float(np.max(per_step))},
        "device": {"name": torch.cuda.get_device_properties(dev).name,
                   "arch": getattr(torch.cuda.get_device_properties(dev), "gcnArchName", ""),
                   "compute_units": torch.cuda.get_device_properties(dev).multi_processor_count,
                   **forward_clock(step, torch, dev, B)},
    }
    out["breakdown"] = breakdown(step, T, H, V, esz, t_act, t_grad, torch)
    if args.timeline:
        vc0 = min(backward_vocab_block(chunk, V, H, esz), V)
        # dH cuts K into pieces when a chunk's token tiles are few (the rule of csrc/layout.hpp)
        pieces = min(max(-(-1024 // (-(-chunk // 256) * -(-H // 256))), 1), 8)
        k_dh = vc0 if pieces == 1 else -(-(-(-vc0 // pieces)) // 64) * 64
        kernels = [("forward", B.KERNEL_HEAD_FORWARD, H)]
        if cfg.backward:
            kernels += [("dz", B.KERNEL_BACKWARD_DZ, H), ("dH", B.KERNEL_BACKWARD_DH, k_dh),
                        ("dW", B.KERNEL_BACKWARD_DW, t_grad if len(chunks) == 1 else None)]
        out["timelines"] = {}
        for name, kid, k in kernels:
            r, khz = kernel_timeline(step, torch, dev, B, kid)
            out["timelines"][name] = timeline_summary(r, khz, k) if khz and r.shape[0] else None
    if args.vendor_gemm:
        log("vendor GEMM (context)")
        vc = backward_vocab_block(chunk, V, H, esz) if cfg.backward else V
        out["vendor_gemm_context"] = vendor_gemm(db, t_act, max(t_grad // len(chunks), 1), vc, torch)
    if not args.no_cpu_baseline:
        log("cpu baseline over " + (f"{args.cpu_rows} rows" if args.cpu_rows > 0 else "a quarter of the rows"))
        out["cpu_baseline"] = cpu_baseline(batch, ref_logp, args.cpu_rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
