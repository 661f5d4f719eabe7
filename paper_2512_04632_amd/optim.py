"""Turbo-Muon as a PyTorch optimizer for matrix parameters.

The paper uses Turbo-Muon as a drop-in replacement for Muon's
orthogonalization and keeps the rest of Muon's step.  This optimizer is a
thin front end of the library's ``tm_muon_step_grouped``: every arithmetic
step (momentum, the bf16 orthogonalization, the parameter update) runs in the
library's kernels; this module only keeps the momentum buffers and passes
pointers.  Parameters must be 2-D fp32 tensors on one GPU (vectors and
scalars belong to another optimizer, as with Muon).
"""
from __future__ import annotations

import torch

from . import _lib


class TurboMuon(torch.optim.Optimizer):
    """Per matrix parameter W with gradient G and momentum buffer M:

        M <- momentum M + G;   U = G + momentum M (nesterov) or M
        W <- W (1 - lr weight_decay) - lr sqrt(max(1, rows/cols)) orthogonalize(U)

    with orthogonalize = ``precond`` pre-conditioning (default AOL) and ``iters``
    quintic Newton-Schulz iterations (default 4) in bf16.
    """

    def __init__(self, params, lr: float = 0.02, momentum: float = 0.95, nesterov: bool = True,
                 weight_decay: float = 0.0, iters: int = 4, precond: str = "aol", coeffs=None,
                 shape_scale: bool = True):
        if lr < 0 or momentum < 0 or weight_decay < 0:
            raise ValueError("lr, momentum and weight_decay must be non-negative")
        defaults = dict(lr=lr, momentum=momentum, nesterov=nesterov, weight_decay=weight_decay,
                        iters=iters, precond=precond, coeffs=coeffs, shape_scale=shape_scale)
        super().__init__(params, defaults)
        for group in self.param_groups:
            for p in group["params"]:
                if p.dim() != 2 or p.dtype != torch.float32:
                    raise ValueError("TurboMuon takes 2-D fp32 parameters only")

    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        for group in self.param_groups:
            ps, gs, ms = [], [], []
            for p in group["params"]:
                if p.grad is None:
                    continue
                state = self.state[p]
                if "momentum_buffer" not in state:
                    state["momentum_buffer"] = torch.zeros_like(p, memory_format=torch.contiguous_format)
                ps.append(p)
                gs.append(p.grad if p.grad.is_contiguous() else p.grad.contiguous())
                ms.append(state["momentum_buffer"])
            if ps:
                _lib.muon_step_grouped(ps, gs, ms, group["lr"], group["momentum"],
                                       group["nesterov"], group["weight_decay"],
                                       group["shape_scale"], group["iters"], group["coeffs"],
                                       group["precond"])
        return loss
