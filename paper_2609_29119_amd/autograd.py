"""Differentiable analysis and synthesis for torch autograd (Sec. 3.2).

Both maps are fixed and real-linear, so no activation is saved: the backward
of each is its explicit real adjoint under <u, v> = Re(u^H v) (eqs. 13-14),
evaluated by the library like the forward maps.

torch's gradient of a real loss with respect to a complex tensor z is
dL/dRe z + i dL/dIm z. For c = T x (x real) the chain rule gives
dL/dx_j = sum_m Re(conj(T_mj) g_m) = (T^dagger g)_j, and for x = S c it gives
the gradient S^dagger g for c; these are NSGCQT_OP_ADJ_ANALYSIS and
NSGCQT_OP_ADJ_SYNTHESIS.
"""
from __future__ import annotations

import torch

from .nsgcqt import OP_ADJ_ANALYSIS, OP_ADJ_SYNTHESIS, Plan


class CQTAnalysis(torch.autograd.Function):
    """c = T x: [batch][N] float32 -> [batch][C] complex64; backward T^dagger."""

    @staticmethod
    def forward(ctx, x, plan: Plan):
        ctx.plan = plan
        return plan.analyse(x.detach().contiguous())

    @staticmethod
    def backward(ctx, grad_c):
        return ctx.plan.adjoint(OP_ADJ_ANALYSIS, grad_c.contiguous()), None


class CQTSynthesis(torch.autograd.Function):
    """x = S c: [batch][C] complex64 -> [batch][N] float32; backward S^dagger."""

    @staticmethod
    def forward(ctx, c, plan: Plan):
        ctx.plan = plan
        return plan.synthesise(c.detach().contiguous())

    @staticmethod
    def backward(ctx, grad_x):
        return ctx.plan.adjoint(OP_ADJ_SYNTHESIS, grad_x.contiguous()), None


def analyse(plan: Plan, x):
    """Differentiable T x."""
    return CQTAnalysis.apply(x, plan)


def synthesise(plan: Plan, c):
    """Differentiable S c."""
    return CQTSynthesis.apply(c, plan)


class CQT(torch.nn.Module):
    """Module wrapper: forward is T, inverse is S, both differentiable."""

    def __init__(self, plan: Plan):
        super().__init__()
        self.plan = plan

    def forward(self, x):
        return analyse(self.plan, x)

    def inverse(self, c):
        return synthesise(self.plan, c)
