"""Write the oracle's per-token log-probs for a full-size synthetic workload.

Usage: python -m tests.golden.make_full_logprobs c2 [c1 c3 c4]

Output: tests/golden/full_<cfg>_logprob.npz with float64 ``logp`` and ``lse``
(0 on rows outside the loss mask). These are the current-policy log-probs of the
seeded batch; the rollout log-probs of that batch are these plus the batch's
drift noise. Only the generator and the oracle are called.
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from synth import CONFIGS, generate  # noqa: E402


def path_for(name: str) -> str:
    return os.path.join(HERE, f"full_{name}_logprob.npz")


def fingerprint(b) -> np.ndarray:
    """A few numbers that change if the generator's draws change."""
    h = b.hidden
    return np.array([b.T, int(b.mask.sum()), int(b.target.astype(np.int64).sum()),
                     float(h[:, 0].astype(np.float64).sum()), float(b.w_head[:, -1].astype(np.float64).sum()),
                     float(b.xi.sum())], dtype=np.float64)


def load(name: str, batch=None):
    """(logp, lse) of a stored workload; checks the fingerprint when a batch is given."""
    d = np.load(path_for(name), allow_pickle=False)
    if batch is not None and not np.array_equal(d["fingerprint"], fingerprint(batch)):
        raise RuntimeError(f"stored oracle values for {name} do not match the generator; "
                           f"rerun python -m tests.golden.make_full_logprobs {name}")
    return d["logp"], d["lse"]


def main(names):
    from oracle import token_logprob  # only the writer runs the oracle; readers of the file do not
    for name in names:
        t0 = time.time()
        b = generate(CONFIGS[name])
        w64 = b.w_head.astype(np.float64)
        logp, lse = token_logprob(b.hidden, None, b.target, b.mask, w64=w64, block=512)
        tmp = path_for(name) + ".tmp.npz"
        np.savez_compressed(tmp, logp=logp, lse=lse, fingerprint=fingerprint(b))
        os.replace(tmp, path_for(name))
        print(f"{name}: {int(b.mask.sum())} rows in {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or ["c2"])
