"""Draft alignment training (AtSpeed-S, Sec. 3.1; AtSpeed-R, Sec. 3.2) of the
draft's item head, driven through atspeed_align_data / atspeed_align_step.

This module holds the buffers the two calls take (the batch, the fp32 master
copy of the head and the AdamW moments) and the learning-rate schedule (the
paper's implementation details: AdamW, lr 1e-3, cosine decay after a linear
warmup).  Every loss, gradient and update runs in the library's kernels.
"""
from __future__ import annotations

import math
from typing import Optional

from .binding import AlignArgs, Engine

MODES = {"S": 0, "R": 1}


def cosine_lr(step: int, total: int, peak: float, warmup: int) -> float:
    """Linear warmup to ``peak`` over ``warmup`` steps, then cosine decay to 0 at ``total``."""
    if warmup > 0 and step <= warmup:
        return peak * step / warmup
    if total <= warmup:
        return peak
    x = min(1.0, (step - warmup) / (total - warmup))
    return 0.5 * peak * (1.0 + math.cos(math.pi * x))


class AlignTrainer:
    """Buffers of one engine's draft-head training.

    ``mode``: "S" (strict verification's objective) or "R" (relaxed); ``alpha``
    the alignment strength (1: the alignment loss alone).  The master copy
    starts from the draft's current item head.
    """

    def __init__(self, eng: Engine, mode: str, alpha: float = 1.0, lr: float = 1e-3, betas=(0.9, 0.999),
                 eps: float = 1e-8, weight_decay: float = 0.01):
        torch = eng.torch
        if eng.draft_dev is None:
            raise ValueError("the engine has no draft model")
        self.eng = eng
        w = eng.w
        B, T, n = eng.cfg.max_batch, eng.max_nodes, eng.n_item
        dev = eng.device
        f32 = dict(dtype=torch.float32, device=dev)
        self.head = eng.draft_dev["lm_head_item"]            # the tensor the draft reads
        d = self.head.shape[1]
        self.ctx_weight = torch.zeros(B * T, **f32)
        self.label_weight = torch.zeros(B * T, **f32)
        self.root_weight = torch.zeros(B, **f32)
        self.log_pK = torch.zeros(B * w.L, **f32)
        self.lp_target = torch.zeros(B * T * n, **f32)
        self.root_target = torch.zeros(B * n, **f32)
        self.master = self.head.float().contiguous().clone()
        self.m = torch.zeros(n * d, **f32)
        self.v = torch.zeros(n * d, **f32)
        self.grad = torch.zeros(n * d, **f32)
        self.args = AlignArgs()
        a = self.args
        a.mode, a.alpha = MODES[mode], alpha
        a.ctx_weight, a.label_weight = self.ctx_weight.data_ptr(), self.label_weight.data_ptr()
        a.root_weight, a.log_pK = self.root_weight.data_ptr(), self.log_pK.data_ptr()
        a.lp_target, a.root_target = self.lp_target.data_ptr(), self.root_target.data_ptr()
        a.master, a.adam_m, a.adam_v, a.grad = (x.data_ptr() for x in (self.master, self.m, self.v, self.grad))
        a.hidden_out = None
        a.lr, a.beta1, a.beta2, a.eps, a.weight_decay = lr, betas[0], betas[1], eps, weight_decay
        a.step = 0

    def data(self, items, n_items, lens=None):
        """The batch of the engine's last prefill: items [B, S, L] int32, n_items [B],
        lens [B, S] (None: whole items) (device)."""
        self.eng.atspeed_align_data(items, lens, n_items, self.args)

    def step(self, lr: Optional[float] = None, hidden_out=None) -> float:
        """One AdamW step; returns the loss before it."""
        a = self.args
        a.step += 1
        if lr is not None:
            a.lr = lr
        a.hidden_out = None if hidden_out is None else hidden_out.data_ptr()
        return self.eng.atspeed_align_step(a)
