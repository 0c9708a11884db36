"""Parity of the whole pass on seeded random small shapes (sizes, vocabularies, element
types, masks, clip widths, GAE settings and the critic), through the C ABI, against the
oracle with the same bars as the fixed cases. The shapes are drawn once from a fixed
seed, so every run checks the same cases."""
import numpy as np
import pytest

from synth import generate, small_config
from tests.gpu_common import compare_all, gpu_pass, oracle_pass, say

pytestmark = pytest.mark.gpu


def _draw_cases(n=12, seed=2607):
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        B = int(rng.integers(1, 10))
        T = int(rng.integers(max(B, 2), 4000))
        H = int(8 * rng.integers(1, 65))
        V = int(rng.integers(1, 6000))
        if T * V * H > 2.5e9:          # keep the fp64 oracle to seconds
            continue
        eps_low = float(rng.choice([0.1, 0.2, 0.3, 0.8]))
        eps_high = float(rng.choice([0.2, 0.28, 3.0, 5.0]))
        a_lo = int(rng.integers(1, 40))
        o_lo = int(rng.integers(1, 40))
        cases.append(dict(
            cfg=dict(name=f"r{len(cases)}", seed=3000 + len(cases), B=B, T=T, H=H, V=V,
                     dtype=str(rng.choice(["bf16", "f32"])), eps_low=eps_low, eps_high=eps_high,
                     xi_sigma=float(rng.choice([0.05, 0.2, 0.5])), act_span=(a_lo, a_lo + int(rng.integers(0, 60))),
                     obs_span=(o_lo, o_lo + int(rng.integers(0, 60))), value_head=bool(rng.random() < 0.3)),
            gamma=float(rng.choice([1.0, 0.99, 0.9])), lam=float(rng.choice([1.0, 0.95, 0.0])),
            alpha=float(rng.choice([0.0, 1.5, 4.0]))))
    return cases


CASES = _draw_cases()


@pytest.mark.parametrize("case", CASES, ids=[c["cfg"]["name"] for c in CASES])
def test_random_shape(case):
    cfg = small_config(**case["cfg"])
    say(f"case {cfg.name}: B={cfg.B} T={cfg.T} H={cfg.H} V={cfg.V} {cfg.dtype} eps={cfg.eps_low}/{cfg.eps_high} "
        f"critic={cfg.value_head} gamma={case['gamma']} lam={case['lam']} alpha={case['alpha']}")
    b = generate(cfg)
    ref = oracle_pass(b, case["gamma"], case["lam"], case["alpha"])
    got = gpu_pass(b, ref["logp"], case["gamma"], case["lam"], case["alpha"])
    compare_all(got, ref, b)
