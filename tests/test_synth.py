"""The seeded generator: shapes, structure, determinism, bf16 rounding, guard band."""
import math

import numpy as np
import pytest
import torch

from synth import CONFIGS, bf16_bits, bf16_round, generate, water_fill
from synth.rollouts import GUARD_DELTA


@pytest.mark.parametrize("name", ["c0", "c1", "c2", "c3", "c4"])
def test_structure(name):
    cfg = CONFIGS[name]
    b = generate(cfg, with_head=(name == "c0"))
    cu = b.cu_seqlens
    assert cu[0] == 0 and (np.diff(cu) >= 1).all() and cu[-1] == b.T
    if cfg.T is not None:
        assert b.T == cfg.T
    assert (b.mask[cu[1:] - 1] == 1).all()                      # last token is an action
    nz = np.nonzero(b.rewards)[0]
    assert set(nz.tolist()) <= set((cu[1:] - 1).tolist())
    assert b.target.min() >= 0 and b.target.max() < cfg.V
    lo = math.log1p(-cfg.eps_low); hi = math.log1p(cfg.eps_high)
    assert np.abs(-b.xi - lo).min() >= GUARD_DELTA and np.abs(-b.xi - hi).min() >= GUARD_DELTA


def test_deterministic_and_head_independent():
    a = generate(CONFIGS["c0"])
    b = generate(CONFIGS["c0"], with_head=False)
    for k in ["cu_seqlens", "mask", "target", "values", "rewards", "xi"]:
        assert np.array_equal(getattr(a, k), getattr(b, k))
    c = generate(CONFIGS["c0"])
    assert np.array_equal(a.hidden, c.hidden) and np.array_equal(a.w_head, c.w_head)


def test_bf16_round_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 3
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 65504.0]   # ties to even
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(bf16_round(x), ref)
    r = bf16_round(x)
    assert np.array_equal(bf16_bits(r), torch.from_numpy(r).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16))


def test_water_fill():
    w = np.array([1.0, 10.0, 100.0, 1000.0])
    L = water_fill(w, 10000, 5000)
    assert L.sum() == 10000 and L.max() <= 5000 and L[3] == 5000
    with pytest.raises(ValueError):
        water_fill(w, 10000, 100)
