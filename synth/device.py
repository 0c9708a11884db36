"""Stage a generated batch in device memory (torch tensors) for the HIP path.

Input staging only: no method arithmetic. The rollout log-probs are a given
reference log-prob plus the batch's drift noise (``rollout_logprobs``).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from .rollouts import Batch, rollout_logprobs


@dataclass
class DeviceBatch:
    hidden: Optional[torch.Tensor]
    w_head: Optional[torch.Tensor]
    target: torch.Tensor
    mask: torch.Tensor
    values: torch.Tensor
    rewards: torch.Tensor
    cu_seqlens: torch.Tensor
    logp_rollout: Optional[torch.Tensor]
    w_value: Optional[torch.Tensor] = None


def head_dtype(batch: Batch) -> torch.dtype:
    return torch.bfloat16 if batch.cfg.dtype == "bf16" else torch.float32


def to_device(batch: Batch, reference_logp: Optional[np.ndarray] = None, device="cuda") -> DeviceBatch:
    dt = head_dtype(batch)

    def mat(x):
        if x is None:
            return None
        return torch.from_numpy(np.ascontiguousarray(x)).to(device=device).to(dt)

    lro = None
    if reference_logp is not None:
        lro = torch.from_numpy(rollout_logprobs(reference_logp, batch.xi)).to(device)
    return DeviceBatch(
        hidden=mat(batch.hidden), w_head=mat(batch.w_head),
        target=torch.from_numpy(batch.target).to(device),
        mask=torch.from_numpy(batch.mask).to(device),
        values=torch.from_numpy(batch.values).to(device),
        rewards=torch.from_numpy(batch.rewards).to(device),
        cu_seqlens=torch.from_numpy(batch.cu_seqlens).to(device),
        logp_rollout=lro, w_value=mat(batch.w_value))
