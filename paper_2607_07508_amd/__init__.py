"""SAO per-token loss pass on AMD MI355X (gfx950): HIP kernels behind a C ABI.

The library (libsao.so, built from csrc/) computes the LM-head log-probs, the
skip-observation GAE advantages, the direct double-sided importance-sampling
loss and its backward, the critic head with its squared-error loss, and the
comparison objectives and critic-free baselines, the step-level GAE and the
explained-variance diagnostic the paper reports. This
package holds the build script and a thin ctypes binding whose functions mirror
the C entry points.
"""
from .binding import (SaoError, advantage, clipped_loss, clipped_loss_noalloc,  # noqa: F401
                      explained_variance, group_advantage, lib, loss_backward, ppo_loss, running_mean_advantage,
                      running_mean_state, step_advantage, token_logprob, value_forward, value_loss, workspace_size)

__version__ = "0.1.0"
