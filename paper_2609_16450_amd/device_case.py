"""Upload a seeded step (workloads.StepCase) to device tensors and wire a StepBuffers."""
from __future__ import annotations

import numpy as np
import torch

from .binding import Ragged, StepBuffers


def _t(x: np.ndarray, dtype: str, device) -> torch.Tensor:
    if dtype == "bf16" and x.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(x)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x)).to(device)


class DeviceStep:
    """Device copies of every input of one step plus freshly allocated outputs."""

    def __init__(self, case, device="cuda", with_max_logit: bool = True):
        dt = case.dtype
        self.case = case
        self.ragged = Ragged(case.batch, case.T, int(case.block_lens.max(initial=0)), case.S,
                             int(case.prefix_lens.max(initial=0)),
                             torch.from_numpy(case.cu_block).to(device),
                             torch.from_numpy(case.cu_prefix).to(device))
        self.q = _t(case.q, dt, device)
        self.k_blk = _t(case.k_blk, dt, device)
        self.v_blk = _t(case.v_blk, dt, device)
        self.k_pre = _t(case.k_pre, dt, device)
        self.v_pre = _t(case.v_pre, dt, device)
        self.h = _t(case.h, dt, device)
        self.w = _t(case.w, dt, device)
        self.tau = torch.from_numpy(case.tau).to(device)
        self.masked0 = torch.from_numpy(case.masked).to(device)
        self.tokens0 = torch.from_numpy(case.tokens).to(device)
        T, B = case.T, case.batch
        self.attn_out = torch.empty_like(self.q)
        self.conf = torch.empty(T, dtype=torch.float32, device=device)
        self.entropy = torch.empty(T, dtype=torch.float32, device=device)
        self.argmax = torch.empty(T, dtype=torch.int32, device=device)
        self.max_logit = torch.empty(T, dtype=torch.float32, device=device) if with_max_logit else None
        self.masked = self.masked0.clone()
        self.tokens = self.tokens0.clone()
        self.unmask = torch.empty(T, dtype=torch.uint8, device=device)
        self.n_commit = torch.empty(B, dtype=torch.int32, device=device)
        self.resolved = torch.empty(B, dtype=torch.uint8, device=device)
        self.buffers = StepBuffers(self.ragged, self.q, self.k_blk, self.v_blk, self.k_pre,
                                   self.v_pre, self.attn_out, self.h, self.w, self.conf,
                                   self.entropy, self.argmax, self.tau, self.masked, self.tokens,
                                   self.unmask, self.n_commit, self.resolved,
                                   max_logit=self.max_logit)

    def reset_state(self) -> None:
        """Restore masked/tokens to the drawn values (the step updates them in place)."""
        self.masked.copy_(self.masked0)
        self.tokens.copy_(self.tokens0)
