"""Seeded synthetic rollout batches for the SAO per-token loss pass.

Each batch stands in for B single rollouts of an agentic task (a math-with-tools
or coding trajectory, paper Sec. 3.2 and Sec. 4.1): model-generated action spans
alternate with environment-observation spans, the last token is an action that
carries a sparse binary terminal reward, and the rollout engine's per-token
log-probs drift from the current policy's by Gaussian noise (Sec. 3.1: the
rollout policy lags the trained one).

Every component draws from its own child stream of ``SeedSequence(seed)`` in a
fixed order (lengths, spans, targets, hidden, W_head and w_value, values,
rewards, drift noise), so a caller may skip the big arrays without changing the
small ones.

Nothing here computes the method: the drift noise is kept away from the two
log-ratios at which the clip band's edges sit (a guard band of width ``delta``),
so that a token's clip decision does not depend on rounding. The rollout
log-probs themselves are built by ``rollout_logprobs`` from a reference log-prob
that the caller supplies.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Optional, Tuple

import numpy as np

__all__ = ["Config", "Batch", "CONFIGS", "generate", "bf16_round", "bf16_bits",
           "rollout_logprobs", "water_fill", "small_config"]

# Guard band on the drift noise around each clip edge (in log-ratio units).
GUARD_DELTA = 4e-3


@dataclass(frozen=True)
class Config:
    """One synthetic workload. Lengths are in tokens."""
    name: str
    seed: int
    B: int
    H: int
    V: int
    dtype: str                      # "f32" or "bf16": element type of hidden and W_head
    length: Tuple                   # ("uniform", lo, hi) | ("lognormal", median, sigma, cap)
                                    # | ("pareto", alpha, x_min, cap)
    T: Optional[int]                # exact total after water-filling (None for "uniform")
    act_span: Tuple[int, int]       # action span length, uniform integer range (inclusive)
    obs_span: Tuple[int, int]       # observation span length, uniform integer range (inclusive)
    value_mean: float
    value_std: float
    reward_p: float                 # Bernoulli probability of reward 1 at the final token
    xi_sigma: float                 # std of the rollout-policy drift noise on log-probs
    eps_low: float
    eps_high: float
    gamma: float = 1.0
    lam: float = 1.0
    alpha: float = 1.5              # length-adaptive lambda; <= 0 means "use lam"
    backward: bool = True
    chunk: Optional[int] = None     # token chunk size of the head pass (None: whole batch)
    value_head: bool = False        # values come from a bias-free H->1 head on hidden
    init_std: float = 0.02


CONFIGS = {
    # Tiny CPU-checkable instance (fp32).
    "c0": Config("c0", 1000, B=4, H=64, V=1000, dtype="f32", length=("uniform", 16, 64), T=None,
                 act_span=(4, 12), obs_span=(2, 8), value_mean=0.5, value_std=0.2, reward_p=0.5,
                 xi_sigma=0.1, eps_low=0.2, eps_high=0.2, alpha=0.0, lam=1.0),
    # Qwen3-30B-A3B head, forward only.
    "c1": Config("c1", 1001, B=16, H=2048, V=151936, dtype="bf16",
                 length=("lognormal", 4096, 0.5, 16384), T=65536,
                 act_span=(800, 2400), obs_span=(64, 2048), value_mean=0.5, value_std=0.2,
                 reward_p=0.5, xi_sigma=0.1, eps_low=0.2, eps_high=0.2, backward=False),
    # Same shapes, forward + backward, larger drift so both clip sides fire.
    "c2": Config("c2", 1002, B=16, H=2048, V=151936, dtype="bf16",
                 length=("lognormal", 4096, 0.5, 16384), T=65536,
                 act_span=(800, 2400), obs_span=(64, 2048), value_mean=0.5, value_std=0.2,
                 reward_p=0.5, xi_sigma=0.2, eps_low=0.2, eps_high=0.2),
    # Long-horizon: heavy-tailed lengths, half the tokens are observations, 8192-token chunks.
    "c3": Config("c3", 1003, B=8, H=2048, V=151936, dtype="bf16",
                 length=("pareto", 1.5, 2048, 65536), T=262144,
                 act_span=(64, 2048), obs_span=(64, 2048), value_mean=0.3, value_std=0.3,
                 reward_p=0.3, xi_sigma=0.1, eps_low=0.2, eps_high=0.2, chunk=8192),
    # Large-MoE head with a scalar value head.
    "c4": Config("c4", 1004, B=64, H=6144, V=151552, dtype="bf16",
                 length=("lognormal", 512, 0.5, 131072), T=32768,
                 act_span=(16, 500), obs_span=(16, 256), value_mean=0.5, value_std=0.2,
                 reward_p=0.5, xi_sigma=0.1, eps_low=0.2, eps_high=0.28, value_head=True),
}


def small_config(name: str, seed: int, B: int, T: int, H: int, V: int, dtype: str = "bf16",
                 **kw) -> Config:
    """A mid-sized variant (many tiles plus ragged tails) for parity tests."""
    base = dict(length=("lognormal", max(8, T // max(B, 1)), 0.5, T), T=T,
                act_span=(8, 40), obs_span=(2, 24), value_mean=0.5, value_std=0.2,
                reward_p=0.5, xi_sigma=0.2, eps_low=0.2, eps_high=0.2)
    base.update(kw)
    return Config(name, seed, B=B, H=H, V=V, dtype=dtype, **base)


@dataclass
class Batch:
    cfg: Config
    cu_seqlens: np.ndarray          # int32 [B+1]
    mask: np.ndarray                # uint8 [T], 1 = model-generated action token
    target: np.ndarray              # int32 [T]
    values: np.ndarray              # float32 [T]
    rewards: np.ndarray             # float32 [T]
    xi: np.ndarray                  # float64 [T], rollout drift noise (guard-banded)
    hidden: Optional[np.ndarray] = None   # float32 [T,H] (bf16-representable when dtype=bf16)
    w_head: Optional[np.ndarray] = None   # float32 [V,H]
    w_value: Optional[np.ndarray] = None  # float32 [H]
    extra: dict = field(default_factory=dict)

    @property
    def T(self) -> int:
        return int(self.mask.shape[0])


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32.

    Finite inputs only: for them the 32-bit sum below cannot wrap.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    flat_x, flat_o = x.reshape(-1).view(np.uint32), out.reshape(-1).view(np.uint32)
    step = 1 << 20
    lsb = np.empty(min(step, flat_x.size), dtype=np.uint32)
    for s in range(0, flat_x.size, step):
        v = flat_x[s:s + step]
        o = flat_o[s:s + step]
        b = lsb[:v.size]
        np.right_shift(v, 16, out=b)
        np.bitwise_and(b, 1, out=b)
        np.add(v, 0x7FFF, out=o)
        np.add(o, b, out=o)
        np.bitwise_and(o, 0xFFFF0000, out=o)
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """The bfloat16 bit patterns of bf16-representable float32 values."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def water_fill(weights: np.ndarray, total: int, cap: int) -> np.ndarray:
    """Integer lengths proportional to ``weights``, each <= cap, summing to ``total``.

    Scale the uncapped weights by a common factor, cap those that overflow and
    repeat; the rounding residue goes to the longest uncapped trajectory.
    """
    w = np.asarray(weights, dtype=np.float64)
    B = w.size
    if B * cap < total:
        raise ValueError("caps cannot hold the requested total")
    capped = np.zeros(B, dtype=bool)
    scaled = w.copy()
    for _ in range(B + 1):
        free = ~capped
        remaining = total - cap * int(capped.sum())
        scaled = np.where(capped, cap, w * (remaining / w[free].sum()))
        over = free & (scaled > cap)
        if not over.any():
            break
        capped |= over
    lengths = np.where(capped, cap, np.floor(scaled)).astype(np.int64)
    lengths = np.maximum(lengths, 1)
    residue = total - int(lengths.sum())
    order = np.argsort(np.where(capped, -1, lengths))[::-1]
    i = 0
    while residue != 0:
        j = order[i % B]
        room = cap - lengths[j] if residue > 0 else lengths[j] - 1
        d = min(abs(residue), room)
        lengths[j] += d if residue > 0 else -d
        residue -= d if residue > 0 else -d
        i += 1
        if i > 4 * B:
            raise RuntimeError("water_fill did not converge")
    assert lengths.sum() == total and lengths.max() <= cap and lengths.min() >= 1
    return lengths


def _lengths(cfg: Config, rng: np.random.Generator) -> np.ndarray:
    kind = cfg.length[0]
    if kind == "uniform":
        _, lo, hi = cfg.length
        return rng.integers(lo, hi + 1, size=cfg.B)
    if kind == "lognormal":
        _, median, sigma, cap = cfg.length
        w = rng.lognormal(mean=math.log(median), sigma=sigma, size=cfg.B)
        return water_fill(w, cfg.T, cap)
    if kind == "pareto":
        _, a, x_min, cap = cfg.length
        w = (rng.pareto(a, size=cfg.B) + 1.0) * x_min
        return water_fill(w, cfg.T, cap)
    raise ValueError(kind)


def _spans(cfg: Config, lengths: np.ndarray, rng: np.random.Generator) -> np.ndarray:
    T = int(lengths.sum())
    mask = np.zeros(T, dtype=np.uint8)
    start = 0
    for L in lengths:
        pos, action = 0, True
        while pos < L:
            lo, hi = cfg.act_span if action else cfg.obs_span
            end = min(pos + int(rng.integers(lo, hi + 1)), int(L))
            if action:
                mask[start + pos:start + end] = 1
            pos, action = end, not action
        mask[start + L - 1] = 1          # the final token is an action: it carries the reward
        start += int(L)
    return mask


def _normal_f32(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    out *= np.float32(std)
    return out


def _guard_banded_noise(cfg: Config, T: int, rng: np.random.Generator,
                        delta: float = GUARD_DELTA) -> np.ndarray:
    # The band edges 1-eps_low and 1+eps_high sit at log-ratios log(1-eps_low) and
    # log(1+eps_high); a rollout log-prob of (reference + xi) gives log-ratio -xi.
    edges = [math.log1p(cfg.eps_high)]
    if cfg.eps_low < 1.0:
        edges.append(math.log1p(-cfg.eps_low))
    xi = rng.normal(0.0, cfg.xi_sigma, size=T)
    for _ in range(1000):
        bad = np.zeros(T, dtype=bool)
        for e in edges:
            bad |= np.abs(-xi - e) < delta
        n = int(bad.sum())
        if n == 0:
            return xi
        xi[bad] = rng.normal(0.0, cfg.xi_sigma, size=n)
    raise RuntimeError("guard band redraw did not terminate")


def generate(cfg: Config, with_head: bool = True) -> Batch:
    """Draw one batch. ``with_head=False`` skips hidden/W (all other arrays are unchanged)."""
    streams = [np.random.Generator(np.random.PCG64(s))
               for s in np.random.SeedSequence(cfg.seed).spawn(8)]
    r_len, r_span, r_tgt, r_hid, r_w, r_val, r_rew, r_xi = streams

    lengths = _lengths(cfg, r_len)
    cu = np.zeros(cfg.B + 1, dtype=np.int64)
    cu[1:] = np.cumsum(lengths)
    T = int(cu[-1])
    mask = _spans(cfg, lengths, r_span)
    target = r_tgt.integers(0, cfg.V, size=T).astype(np.int32)

    hidden = w_head = w_value = None
    if with_head:
        hidden = _normal_f32(r_hid, (T, cfg.H), cfg.init_std)
        w_head = _normal_f32(r_w, (cfg.V, cfg.H), cfg.init_std)
        if cfg.value_head:
            w_value = _normal_f32(r_w, (cfg.H,), cfg.init_std)
        if cfg.dtype == "bf16":
            hidden = bf16_round(hidden)
            w_head = bf16_round(w_head)
            if w_value is not None:
                w_value = bf16_round(w_value)

    values = (cfg.value_mean + cfg.value_std * r_val.standard_normal(T)).astype(np.float32)
    rewards = np.zeros(T, dtype=np.float32)
    rewards[cu[1:] - 1] = (r_rew.random(cfg.B) < cfg.reward_p).astype(np.float32)
    xi = _guard_banded_noise(cfg, T, r_xi)
    return Batch(cfg=cfg, cu_seqlens=cu.astype(np.int32), mask=mask, target=target,
                 values=values, rewards=rewards, xi=xi, hidden=hidden, w_head=w_head,
                 w_value=w_value)


def rollout_logprobs(reference_logp: np.ndarray, xi: np.ndarray) -> np.ndarray:
    """The rollout engine's recorded log-probs: a reference log-prob plus drift noise."""
    return (np.asarray(reference_logp, dtype=np.float64) + xi).astype(np.float32)


def comparison_logprobs(cfg: Config, T: int, behav_sigma: float = 0.05):
    """Per-token log-probs for the comparison objectives, all float32 [T]:
    the current policy's (exponentially spread below 0), the old policy's (the
    current ones plus guard-banded drift noise, so every log-ratio stays clear of
    the clip edges of cfg) and the rollout engine's (the old ones plus small noise)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, 7919])))
    lp = (-rng.exponential(1.0, T)).astype(np.float32)
    lold = rollout_logprobs(lp, _guard_banded_noise(cfg, T, rng))
    lb = (lold.astype(np.float64) + rng.normal(0.0, behav_sigma, T)).astype(np.float32)
    return lp, lold, lb


def with_overrides(cfg: Config, **kw) -> Config:
    return replace(cfg, **kw)
