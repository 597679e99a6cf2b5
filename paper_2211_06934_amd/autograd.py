"""torch.autograd.Functions around the fused differentiable optimizer steps.

Mirrors Listing 1's functional API: ``opt.init`` creates (mu, nu, count);
``opt.update(grads, state, inplace=False)`` followed by ``apply_updates`` is
one call of AdamFn, whose backward is the library's VJP kernel (Sec. 2.3:
the optimizer as one operator with a hand-written backward).  The Function
only allocates outputs and forwards pointers to the C ABI.

Every backward here is a kernel with no autograd graph of its own, so the
Functions are differentiable once (``once_differentiable``): a first-order
meta-gradient through any number of unrolled steps works, and asking for a
higher-order one (``create_graph=True`` through a fused step) raises an error
instead of silently treating the VJP's inputs as constants.
"""
from __future__ import annotations

import dataclasses

import torch
from torch.autograd.function import once_differentiable

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
    @once_differentiable
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
        from .tree import leaf_pointer_tensors
        S = len(leaves) // 4
        p, g, m, v = (list(leaves[i * S:(i + 1) * S]) for i in range(4))
        p, g, m, v = ([x.contiguous() for x in t] for t in (p, g, m, v))
        dev = p[0].device
        po = [torch.empty_like(x) for x in p]
        mo = [torch.empty_like(x) for x in m]
        vo = [torch.empty_like(x) for x in v]
        ptr = leaf_pointer_tensors((p, g, m, v, po, mo, vo), dev)
        _d.adam_fwd_tree(table, ptr[0], ptr[1], ptr[2], ptr[3], count, hyper.lr, hyper.b1, hyper.b2, hyper.eps,
                         hyper.eps_root, ptr[4], ptr[5], ptr[6])
        ctx.save_for_backward(*g, *m, *v)
        ctx.S, ctx.count, ctx.hyper, ctx.table = S, count, hyper, table
        return (*po, *mo, *vo)

    @staticmethod
    @once_differentiable
    def backward(ctx, *cots):
        from .tree import leaf_pointer_tensors
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
        ptr = leaf_pointer_tensors((dP, dM, dV, g, m, v, dg, dm, dv), dev)
        _d.adam_bwd_tree(ctx.table, ptr[0], ptr[1], ptr[2], ptr[3], ptr[4], ptr[5], ctx.count, h.lr, h.b1, h.b2,
                         h.eps, h.eps_root, ptr[6], ptr[7], ptr[8])
        # the params path is the identity: the cotangent of each p leaf is dP
        return (None, None, None, *dP, *dg, *dm, *dv)


class _MetaOptimizer:
    """Module-parameter plumbing shared by the object-oriented optimizers
    (Listing 1, OOP API): the trainable parameters in registration order, one
    cached segment table for their shapes, and the installation of updated,
    non-leaf tensors as the module's parameters."""

    def __init__(self, module: torch.nn.Module):
        from .tree import segment_table
        self.module = module
        self.names = [n for n, p in module.named_parameters() if p.requires_grad]
        if not self.names:
            raise ValueError("the module has no trainable parameters")
        params = [self._get(n) for n in self.names]
        if any(p.dtype != torch.float32 or p.device != params[0].device for p in params):
            raise ValueError("the fused optimizers take fp32 parameters on one device")
        self.table = segment_table([tuple(p.shape) for p in params], params[0].dtype, params[0].device)

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

    def _install(self, new_params) -> None:
        for name, p in zip(self.names, new_params):
            self._set(name, p)

    def _detach_params(self) -> None:
        for name in self.names:
            p = self._get(name)
            self._set(name, torch.nn.Parameter(p.detach().clone()) if not isinstance(p, torch.nn.Parameter) else p)


class MetaAdam(_MetaOptimizer):
    """Object-oriented differentiable Adam over a module's parameters
    (Listing 1, OOP API: ``opt = MetaAdam(model); opt.step(loss)``).

    Each step differentiates the loss w.r.t. the current parameters with
    create_graph=True, applies one leaf-direct fused Adam step (AdamTreeFn) and
    installs the updated, non-leaf tensors as the module's parameters, so a
    later outer loss backpropagates through every inner step (explicit
    gradient).  ``detach_()`` cuts the graph, e.g. between outer iterations.
    """

    def __init__(self, module: torch.nn.Module, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, eps_root=0.0):
        super().__init__(module)
        self.hyper = AdamHyper(lr, b1, b2, eps, eps_root)
        params = self.params()
        self.mu = [torch.zeros_like(p) for p in params]
        self.nu = [torch.zeros_like(p) for p in params]
        self.count = 0

    def step(self, loss: torch.Tensor) -> None:
        params = self.params()
        grads = torch.autograd.grad(loss, params, create_graph=True)
        out = AdamTreeFn.apply(self.table, self.count, self.hyper, *params, *grads, *self.mu, *self.nu)
        S = len(params)
        self._install(out[:S])
        self.mu, self.nu = list(out[S:2 * S]), list(out[2 * S:])
        self.count += 1

    def detach_(self) -> None:
        self._detach_params()
        self.mu = [m.detach() for m in self.mu]
        self.nu = [v.detach() for v in self.nu]


# ---- SGD-momentum and RMSProp (the paper's other fused optimizers) ------------------


@dataclasses.dataclass(frozen=True)
class SGDHyper:
    lr: float = 0.1
    momentum: float = 0.0
    nesterov: bool = False


@dataclasses.dataclass(frozen=True)
class RMSPropHyper:
    lr: float = 1e-2
    alpha: float = 0.99
    eps: float = 1e-8
    eps_root: float = 0.0
    momentum: float = 0.0


def _ptrs(groups, dev):
    from .tree import leaf_pointer_tensors
    return leaf_pointer_tensors(groups, dev)


class SGDTreeFn(torch.autograd.Function):
    """Leaf-direct differentiable SGD step (momentum, Nesterov optional).

    apply(table, hyper, has_trace, *leaves) with leaves = p_1..p_S, g_1..g_S
    and, when has_trace, the trace t_1..t_S; returns p'_1..p'_S and, when
    momentum > 0, t'_1..t'_S.  The VJP is linear in the cotangents, so nothing
    is saved; absent cotangents go to the kernel as NULL (zero)."""

    @staticmethod
    def forward(ctx, table, hyper: SGDHyper, has_trace: bool, *leaves):
        S = len(table.numel)
        p, g = [x.contiguous() for x in leaves[:S]], [x.contiguous() for x in leaves[S:2 * S]]
        t = [x.contiguous() for x in leaves[2 * S:3 * S]] if has_trace else None
        mom = hyper.momentum > 0
        dev = p[0].device
        po = [torch.empty_like(x) for x in p]
        to = [torch.empty_like(x) for x in p] if mom else None
        a = _ptrs((p, g, t, po, to), dev)
        _d.sgd_fwd_tree(table, a[0], a[1], a[2], hyper.lr, hyper.momentum, hyper.nesterov, a[3], a[4])
        ctx.table, ctx.hyper, ctx.has_trace, ctx.S = table, hyper, has_trace, S
        ctx.shapes, ctx.dtype, ctx.device = [x.shape for x in p], p[0].dtype, dev
        return (*po, *to) if mom else tuple(po)

    @staticmethod
    @once_differentiable
    def backward(ctx, *cots):
        S, h = ctx.S, ctx.hyper
        mom = h.momentum > 0
        dev = ctx.device
        new = lambda shape: torch.empty(shape, dtype=ctx.dtype, device=dev)  # noqa: E731
        zero = lambda shape: torch.zeros(shape, dtype=ctx.dtype, device=dev)  # noqa: E731
        dP = [zero(sh) if c is None else c.contiguous() for c, sh in zip(cots[:S], ctx.shapes)]
        dT = None
        if mom and any(c is not None for c in cots[S:2 * S]):
            dT = [zero(sh) if c is None else c.contiguous() for c, sh in zip(cots[S:2 * S], ctx.shapes)]
        dg = [new(sh) for sh in ctx.shapes]
        dt = [new(sh) for sh in ctx.shapes] if mom else None
        a = _ptrs((dP, dT, dg, dt), dev)
        _d.sgd_bwd_tree(ctx.table, a[0], a[1], h.lr, h.momentum, h.nesterov, a[2], a[3])
        # the params path is the identity: the cotangent of each p leaf is dP
        grads = [*dP, *dg]
        if ctx.has_trace:
            grads += dt if mom else [None] * S
        return (None, None, None, *grads)


class RMSPropTreeFn(torch.autograd.Function):
    """Leaf-direct differentiable RMSProp step (momentum optional).

    apply(table, hyper, has_mom, *leaves) with leaves = p_1..p_S, g_1..g_S,
    v_1..v_S and, when has_mom, the momentum buffer b_1..b_S; returns
    p'_1..p'_S, v'_1..v'_S and, when momentum > 0, b'_1..b'_S.  The VJP
    (reduced form, Sec. 2.3) uses the saved g and v."""

    @staticmethod
    def forward(ctx, table, hyper: RMSPropHyper, has_mom: bool, *leaves):
        S = len(table.numel)
        p, g, v = ([x.contiguous() for x in leaves[i * S:(i + 1) * S]] for i in range(3))
        b = [x.contiguous() for x in leaves[3 * S:4 * S]] if has_mom else None
        mom = hyper.momentum > 0
        dev = p[0].device
        po = [torch.empty_like(x) for x in p]
        vo = [torch.empty_like(x) for x in v]
        bo = [torch.empty_like(x) for x in p] if mom else None
        h = hyper
        a = _ptrs((p, g, v, b, po, vo, bo), dev)
        _d.rmsprop_fwd_tree(table, a[0], a[1], a[2], a[3], h.lr, h.alpha, h.eps, h.eps_root, h.momentum, a[4], a[5],
                            a[6])
        ctx.save_for_backward(*g, *v)
        ctx.table, ctx.hyper, ctx.has_mom, ctx.S = table, hyper, has_mom, S
        return (*po, *vo, *bo) if mom else (*po, *vo)

    @staticmethod
    @once_differentiable
    def backward(ctx, *cots):
        S, h = ctx.S, ctx.hyper
        mom = h.momentum > 0
        saved = ctx.saved_tensors
        g, v = saved[:S], saved[S:]
        dev = g[0].device

        def cot(group):
            if all(c is None for c in group):
                return None
            return [torch.zeros_like(x) if c is None else c.contiguous() for c, x in zip(group, g)]

        dP = cot(cots[:S]) or [torch.zeros_like(x) for x in g]
        dV = cot(cots[S:2 * S])
        dB = cot(cots[2 * S:3 * S]) if mom else None
        dg = [torch.empty_like(x) for x in g]
        dv = [torch.empty_like(x) for x in v]
        db = [torch.empty_like(x) for x in g] if mom else None
        a = _ptrs((dP, dV, dB, g, v, dg, dv, db), dev)
        _d.rmsprop_bwd_tree(ctx.table, a[0], a[1], a[2], a[3], a[4], h.lr, h.alpha, h.eps, h.eps_root, h.momentum,
                            a[5], a[6], a[7])
        grads = [*dP, *dg, *dv]
        if ctx.has_mom:
            grads += db if mom else [None] * S
        return (None, None, None, *grads)


class MetaSGD(_MetaOptimizer):
    """Object-oriented differentiable SGD (momentum, Nesterov optional) over a
    module's parameters; each step is one leaf-direct launch (SGDTreeFn).  The
    trace starts absent (zero), as torch.optim's first momentum step."""

    def __init__(self, module: torch.nn.Module, lr=0.1, momentum=0.0, nesterov=False):
        super().__init__(module)
        self.hyper = SGDHyper(lr, momentum, nesterov)
        self.trace = None

    def step(self, loss: torch.Tensor) -> None:
        params = self.params()
        grads = torch.autograd.grad(loss, params, create_graph=True)
        has_trace = self.trace is not None
        out = SGDTreeFn.apply(self.table, self.hyper, has_trace, *params, *grads, *(self.trace or []))
        S = len(params)
        self._install(out[:S])
        if self.hyper.momentum > 0:
            self.trace = list(out[S:])

    def detach_(self) -> None:
        self._detach_params()
        if self.trace is not None:
            self.trace = [t.detach() for t in self.trace]


class MetaRMSProp(_MetaOptimizer):
    """Object-oriented differentiable RMSProp (momentum optional) over a
    module's parameters; each step is one leaf-direct launch (RMSPropTreeFn)."""

    def __init__(self, module: torch.nn.Module, lr=1e-2, alpha=0.99, eps=1e-8, eps_root=0.0, momentum=0.0):
        super().__init__(module)
        self.hyper = RMSPropHyper(lr, alpha, eps, eps_root, momentum)
        self.nu = [torch.zeros_like(p) for p in self.params()]
        self.mom = None

    def step(self, loss: torch.Tensor) -> None:
        params = self.params()
        grads = torch.autograd.grad(loss, params, create_graph=True)
        has_mom = self.mom is not None
        out = RMSPropTreeFn.apply(self.table, self.hyper, has_mom, *params, *grads, *self.nu, *(self.mom or []))
        S = len(params)
        self._install(out[:S])
        self.nu = list(out[S:2 * S])
        if self.hyper.momentum > 0:
            self.mom = list(out[2 * S:])

    def detach_(self) -> None:
        self._detach_params()
        self.nu = [v.detach() for v in self.nu]
        if self.mom is not None:
            self.mom = [b.detach() for b in self.mom]


def es_gradient(fn, theta: torch.Tensor, sigma: float, num_samples: int, method: str = "antithetic",
                seed: int = None, sample=None) -> torch.Tensor:
    """Zero-order (ES) estimate of the gradient of the Gaussian smoothing of fn
    at theta (Sec. 2.2).  fn maps a batch [M, n] to [M] and is evaluated once
    on all perturbed points (and once on theta for the baseline method).

    By default the N(0, I) noise is generated inside the kernels from `seed`
    (a 64-bit integer; drawn from torch's CPU generator when None): the
    perturbed points come from diffopt_es_perturb_gaussian and the estimate
    from diffopt_es_estimate_gaussian, which forms the method's weights from
    the evaluations, so no noise array exists.  `sample`, a callable
    (num_samples, n) -> [num_samples, n] device tensor, draws the noise from
    another distribution instead (Listing 3's customisable sampler); then the
    explicit-noise kernels run, with the weights formed by diffopt_es_weights.
    method: "plain", "baseline" (subtract f(theta)) or "antithetic"."""
    if method not in _d.ES_METHODS:
        raise ValueError("method must be plain, baseline or antithetic")
    theta = theta.detach().contiguous().reshape(-1)
    n = theta.numel()
    anti = method == "antithetic"
    pts = torch.empty((2 if anti else 1) * num_samples, n, device=theta.device, dtype=theta.dtype)
    noise = None
    if sample is None:
        if seed is None:
            seed = int(torch.randint(0, 2 ** 62, (1,)).item())
        _d.es_perturb_gaussian(theta, num_samples, seed, sigma, anti, pts)
    else:
        noise = sample(num_samples, n)
        if tuple(noise.shape) != (num_samples, n):
            raise ValueError("sample must return a [num_samples, n] tensor")
        noise = noise.to(device=theta.device, dtype=theta.dtype).contiguous()
        _d.es_perturb(theta, noise, sigma, anti, pts)
    with torch.no_grad():
        fv = fn(pts).reshape(-1).to(theta.dtype).contiguous()
        f0 = fn(theta.reshape(1, -1)).reshape(1).to(theta.dtype).contiguous() if method == "baseline" else None
    grad = torch.empty_like(theta)
    if noise is None:
        _d.es_estimate_gaussian(fv, method, num_samples, seed, sigma, grad, f0=f0)
    else:
        w = torch.empty(num_samples, device=theta.device, dtype=theta.dtype)
        _d.es_weights(fv, method, num_samples, sigma, w, f0=f0)
        _d.es_estimate(noise, w, 1.0, grad)
    return grad


class ZeroOrderFn(torch.autograd.Function):
    """y = fn(theta) whose backward is the ES gradient estimate (Sec. 2.2,
    the zero_order decorator's behaviour): grad_theta = grad_y * estimate.
    apply(theta, fn, sigma, num_samples, method, seed[, sample])."""

    @staticmethod
    def forward(ctx, theta, fn, sigma, num_samples, method, seed=None, sample=None):
        ctx.save_for_backward(theta)
        ctx.cfg = (fn, sigma, num_samples, method, seed, sample)
        with torch.no_grad():
            return fn(theta.detach().reshape(1, -1)).reshape(())

    @staticmethod
    @once_differentiable
    def backward(ctx, grad_y):
        (theta,) = ctx.saved_tensors
        fn, sigma, num_samples, method, seed, sample = ctx.cfg
        g = es_gradient(fn, theta, sigma, num_samples, method, seed, sample).reshape(theta.shape)
        return grad_y * g, None, None, None, None, None, None
