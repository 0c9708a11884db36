"""Seeded synthetic single-rollout batches shaped like the paper's agentic workloads.

This package only draws inputs. It holds none of the method's arithmetic:
no log-softmax, no advantage, no ratio. Both the fp64 oracle and the HIP
path read the arrays it returns.
"""
from .rollouts import (CONFIGS, Config, Batch, generate, bf16_round, bf16_bits,  # noqa: F401
                       rollout_logprobs, small_config, water_fill, with_overrides,
                       comparison_logprobs)
