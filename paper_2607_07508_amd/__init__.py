"""SAO per-token loss pass on AMD MI355X (gfx950): HIP kernels behind a C ABI.

The library (libsao.so, built from csrc/) computes the LM-head log-probs, the
skip-observation GAE advantages, the direct double-sided importance-sampling
loss and its backward, and the critic head with its squared-error loss. This
package holds the build script and a thin ctypes binding whose functions mirror
the C entry points.
"""
from .binding import (SaoError, advantage, clipped_loss, lib, loss_backward,  # noqa: F401
                      token_logprob, value_forward, value_loss, workspace_size)

__version__ = "0.1.0"
