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


class AdamTreeFn(torch.autograd.Function):
    """Leaf-direct differentiable Adam step over a list of fp32 leaves.

    apply(table, count, hyper, *leaves) with leaves = p_1..p_S, g_1..g_S,
    m_1..m_S, v_1..v_S returns p'_1..p'_S, m'_1..m'_S, v'_1..v'_S.  Forward and
    backward are single launches of the tree-map kernels over the segment table
    (no flatten); the leaf-address arrays are built per call.
    """

    @staticmethod
    def forward(ctx, table, count: int, hyper: AdamHyper, *leaves):
        from .tree import leaf_pointer_tensor
        S = len(leaves) // 4
        p, g, m, v = (list(leaves[i * S:(i + 1) * S]) for i in range(4))
        p, g, m, v = ([x.contiguous() for x in t] for t in (p, g, m, v))
        dev = p[0].device
        po = [torch.empty_like(x) for x in p]
        mo = [torch.empty_like(x) for x in m]
        vo = [torch.empty_like(x) for x in v]
        ptr = [leaf_pointer_tensor(t, dev) for t in (p, g, m, v, po, mo, vo)]
        _d.adam_fwd_tree(table, ptr[0], ptr[1], ptr[2], ptr[3], count, hyper.lr, hyper.b1, hyper.b2, hyper.eps,
                         hyper.eps_root, ptr[4], ptr[5], ptr[6])
        ctx.save_for_backward(*g, *m, *v)
        ctx.S, ctx.count, ctx.hyper, ctx.table = S, count, hyper, table
        return (*po, *mo, *vo)

    @staticmethod
    def backward(ctx, *cots):
        from .tree import leaf_pointer_tensor
        S, h = ctx.S, ctx.hyper
        saved = ctx.saved_tensors
        g, m, v = saved[:S], saved[S:2 * S], saved[2 * S:]
        dev = g[0].device
        dP = [torch.zeros_like(x) if c is None else c.contiguous() for c, x in zip(cots[:S], g)]
        dM = [torch.zeros_like(x) if c is None else c.contiguous() for c, x in zip(cots[S:2 * S], m)]
        dV = [torch.zeros_like(x) if c is None else c.contiguous() for c, x in zip(cots[2 * S:], v)]
        dg = [torch.empty_like(x) for x in g]
        dm = [torch.empty_like(x) for x in m]
        dv = [torch.empty_like(x) for x in v]
        ptr = [leaf_pointer_tensor(t, dev) for t in (dP, dM, dV, g, m, v, dg, dm, dv)]
        _d.adam_bwd_tree(ctx.table, ptr[0], ptr[1], ptr[2], ptr[3], ptr[4], ptr[5], ctx.count, h.lr, h.b1, h.b2,
                         h.eps, h.eps_root, ptr[6], ptr[7], ptr[8])
        # the params path is the identity: the cotangent of each p leaf is dP
        return (None, None, None, *dP, *dg, *dm, *dv)


class MetaAdam:
    """Object-oriented differentiable Adam over a module's parameters
    (Listing 1, OOP API: ``opt = MetaAdam(model); opt.step(loss)``).

    Each step differentiates the loss w.r.t. the current parameters with
    create_graph=True, applies one leaf-direct fused Adam step (AdamTreeFn) and
    installs the updated, non-leaf tensors as the module's parameters, so a
    later outer loss backpropagates through every inner step (explicit
    gradient).  ``detach_()`` cuts the graph, e.g. between outer iterations.
    """

    def __init__(self, module: torch.nn.Module, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, eps_root=0.0):
        from .tree import segment_table
        self.module = module
        self.hyper = AdamHyper(lr, b1, b2, eps, eps_root)
        self.names = [n for n, p in module.named_parameters() if p.requires_grad]
        params = [self._get(n) for n in self.names]
        self.table = segment_table([tuple(p.shape) for p in params], params[0].dtype, params[0].device)
        self.mu = [torch.zeros_like(p) for p in params]
        self.nu = [torch.zeros_like(p) for p in params]
        self.count = 0

    def _owner(self, name):
        mod = self.module
        *path, leaf = name.split(".")
        for part in path:
            mod = getattr(mod, part)
        return mod, leaf

    def _get(self, name):
        mod, leaf = self._owner(name)
        return mod._parameters[leaf]

    def _set(self, name, value):
        mod, leaf = self._owner(name)
        mod._parameters[leaf] = value

    def params(self):
        return [self._get(n) for n in self.names]

    def step(self, loss: torch.Tensor) -> None:
        params = self.params()
        grads = torch.autograd.grad(loss, params, create_graph=True)
        out = AdamTreeFn.apply(self.table, self.count, self.hyper, *params, *grads, *self.mu, *self.nu)
        S = len(params)
        for name, p in zip(self.names, out[:S]):
            self._set(name, p)
        self.mu, self.nu = list(out[S:2 * S]), list(out[2 * S:])
        self.count += 1

    def detach_(self) -> None:
        for name in self.names:
            p = self._get(name)
            self._set(name, torch.nn.Parameter(p.detach().clone()) if not isinstance(p, torch.nn.Parameter) else p)
        self.mu = [m.detach() for m in self.mu]
        self.nu = [v.detach() for v in self.nu]


def es_gradient(fn, theta: torch.Tensor, sigma: float, num_samples: int, method: str = "antithetic",
                generator: torch.Generator = None) -> torch.Tensor:
    """Zero-order (ES) estimate of the gradient of the Gaussian smoothing of fn
    at theta (Sec. 2.2): draws N(0, I) noise with the caller's generator,
    builds the perturbed points with diffopt_es_perturb, evaluates fn on them
    as one batch (fn maps [M, n] to [M]) and reduces with diffopt_es_estimate.
    method: "plain", "baseline" (subtract f(theta)) or "antithetic"."""
    if method not in ("plain", "baseline", "antithetic"):
        raise ValueError("method must be plain, baseline or antithetic")
    theta = theta.detach().contiguous().reshape(-1)
    n = theta.numel()
    noise = torch.randn(num_samples, n, device=theta.device, dtype=theta.dtype, generator=generator)
    anti = method == "antithetic"
    pts = torch.empty((2 if anti else 1) * num_samples, n, device=theta.device, dtype=theta.dtype)
    _d.es_perturb(theta, noise, sigma, anti, pts)
    with torch.no_grad():
        fv = fn(pts).reshape(-1).to(theta.dtype)
        if method == "plain":
            w, scale = fv, 1.0 / (num_samples * sigma)
        elif method == "baseline":
            w, scale = fv - fn(theta.reshape(1, -1)).reshape(()), 1.0 / (num_samples * sigma)
        else:
            w, scale = fv[:num_samples] - fv[num_samples:], 1.0 / (2 * num_samples * sigma)
    grad = torch.empty_like(theta)
    _d.es_estimate(noise, w.contiguous(), scale, grad)
    return grad


class ZeroOrderFn(torch.autograd.Function):
    """y = fn(theta) whose backward is the ES gradient estimate (Sec. 2.2,
    the zero_order decorator's behaviour): grad_theta = grad_y * estimate."""

    @staticmethod
    def forward(ctx, theta, fn, sigma, num_samples, method, generator):
        ctx.save_for_backward(theta)
        ctx.cfg = (fn, sigma, num_samples, method, generator)
        with torch.no_grad():
            return fn(theta.detach().reshape(1, -1)).reshape(())

    @staticmethod
    def backward(ctx, grad_y):
        (theta,) = ctx.saved_tensors
        fn, sigma, num_samples, method, generator = ctx.cfg
        g = es_gradient(fn, theta, sigma, num_samples, method, generator).reshape(theta.shape)
        return grad_y * g, None, None, None, None, None
