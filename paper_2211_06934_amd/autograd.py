"""torch.autograd.Function around the fused differentiable Adam step.

Mirrors Listing 1's functional API: ``opt.init`` creates (mu, nu, count);
``opt.update(grads, state, inplace=False)`` followed by ``apply_updates`` is
one call of AdamFn, whose backward is the library's VJP kernel (Sec. 2.3:
the optimizer as one operator with a hand-written backward).  The Function
only allocates outputs and forwards pointers to the C ABI.
"""
from __future__ import annotations

import dataclasses

import torch

from . import diffopt as _d


@dataclasses.dataclass
class AdamState:
    mu: torch.Tensor
    nu: torch.Tensor
    count: int


@dataclasses.dataclass(frozen=True)
class AdamHyper:
    lr: float = 1e-3
    b1: float = 0.9
    b2: float = 0.999
    eps: float = 1e-8
    eps_root: float = 0.0


class AdamFn(torch.autograd.Function):
    """(p, g, m, v) -> (p', m', v') for one differentiable Adam step on flat fp32 buffers."""

    @staticmethod
    def forward(ctx, p, g, m, v, count: int, hyper: AdamHyper):
        p, g, m, v = (x.contiguous() for x in (p, g, m, v))
        po, mo, vo = torch.empty_like(p), torch.empty_like(m), torch.empty_like(v)
        _d.adam_fwd(p, g, m, v, count, hyper.lr, hyper.b1, hyper.b2, hyper.eps, hyper.eps_root,
                    po, mo, vo)
        ctx.save_for_backward(g, m, v)
        ctx.count = count
        ctx.hyper = hyper
        return po, mo, vo

    @staticmethod
    def backward(ctx, dP, dM, dV):
        g, m, v = ctx.saved_tensors
        h = ctx.hyper
        if dP is None:
            dP = torch.zeros_like(g)
        dP = dP.contiguous()
        if dM is None and dV is None:
            dM_in = dV_in = None
        else:
            dM_in = torch.zeros_like(m) if dM is None else dM.contiguous()
            dV_in = torch.zeros_like(v) if dV is None else dV.contiguous()
        dg, dm, dv = torch.empty_like(g), torch.empty_like(m), torch.empty_like(v)
        _d.adam_bwd(dP, dM_in, dV_in, g, m, v, ctx.count, h.lr, h.b1, h.b2, h.eps, h.eps_root,
                    None, dg, dm, dv)
        # the params path is the identity: the cotangent of p is dP itself
        return dP, dg, dm, dv, None, None


class FlatAdam:
    """Functional differentiable Adam over one flat buffer (Listing 1, functional API)."""

    def __init__(self, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, eps_root=0.0):
        self.hyper = AdamHyper(lr, b1, b2, eps, eps_root)

    def init(self, params: torch.Tensor) -> AdamState:
        return AdamState(torch.zeros_like(params), torch.zeros_like(params), 0)

    def step(self, params: torch.Tensor, grads: torch.Tensor, state: AdamState):
        """Non-inplace update fused with apply_updates; differentiable."""
        p, m, v = AdamFn.apply(params, grads, state.mu, state.nu, state.count, self.hyper)
        return p, AdamState(m, v, state.count + 1)
