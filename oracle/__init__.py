"""Plain fp64 CPU oracle of the SAO per-token loss pass.

TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this package. The product path (the
HIP library and its Python binding) never imports it and has no CPU fallback.
"""
from .sao_oracle import (  # noqa: F401
    token_logprob, token_logprob_loop, advantage, dis_loss,
    loss_backward, loss_backward_loop, value_forward, value_loss, surrogate_S,
    ppo_loss, explained_variance, step_advantage, steps_of,
    trajectory_rewards, group_advantage, running_mean_advantage,
)
