"""Pins of the oracle's fused SGD-momentum and RMSProp steps and their VJPs:
closed forms, torch.optim's SGD / RMSprop in fp64 (library routines, forward
over many steps and autograd through their functional forms), central
differences, and the symmetric derivative at RMSProp's 0/0 point."""
import numpy as np
import pytest
import torch

import oracle
from workloads import abs_normal, normal


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b) / np.maximum(np.abs(b), 1e-300)))


# ------------------------------------------------------------------- SGD


@pytest.mark.parametrize("momentum,nesterov", [(0.0, False), (0.9, False), (0.9, True), (0.5, True)])
def test_sgd_matches_torch_optim_over_steps(momentum, nesterov):
    n, K, lr = 500, 12, 0.05
    p0 = normal(n, 0.05, "sgd", "p0").astype(np.float64)
    grads = [normal(n, 0.01, "sgd", "grad", k).astype(np.float64) for k in range(K)]
    p, t = p0, None
    for g in grads:
        p, t1 = oracle.sgd_fwd(p, g, t, lr, momentum, nesterov)
        t = t1 if momentum > 0 else None
    tp = torch.tensor(p0, requires_grad=True)
    opt = torch.optim.SGD([tp], lr=lr, momentum=momentum, nesterov=nesterov, dampening=0.0)
    for g in grads:
        tp.grad = torch.tensor(g)
        opt.step()
    assert _rel(p - p0, tp.detach().numpy() - p0) < 1e-12


def test_sgd_plain_closed_form_and_trace():
    n = 100
    p = normal(n, 0.05, "sgd", "p0", 1).astype(np.float64)
    g = normal(n, 0.01, "sgd", "grad", 1).astype(np.float64)
    t = normal(n, 0.01, "sgd", "mu", 1).astype(np.float64)
    po, to = oracle.sgd_fwd(p, g, None, 0.1)
    assert np.array_equal(po, p - 0.1 * g) and np.array_equal(to, g)
    po, to = oracle.sgd_fwd(p, g, t, 0.1, 0.9)
    assert _rel(to, 0.9 * t + g) < 1e-15 and _rel(po, p - 0.1 * (0.9 * t + g)) < 1e-15


@pytest.mark.parametrize("momentum,nesterov", [(0.0, False), (0.9, False), (0.9, True)])
def test_sgd_vjp_matches_torch_autograd(momentum, nesterov):
    from torch.optim.sgd import sgd
    n, lr = 300, 0.05
    p = torch.tensor(normal(n, 0.05, "sgd", "p0", 2).astype(np.float64), requires_grad=True)
    g = torch.tensor(normal(n, 0.01, "sgd", "grad", 2).astype(np.float64), requires_grad=True)
    t = torch.tensor(normal(n, 0.01, "sgd", "mu", 2).astype(np.float64), requires_grad=True)
    cP = normal(n, 1.0, "sgd", "cot_p", 2).astype(np.float64)
    cT = normal(n, 1.0, "sgd", "cot_m", 2).astype(np.float64)
    pc, gc, tc = p.clone(), g.clone(), t.clone()
    # a zero-or-given buffer keeps torch's first step differentiable
    sgd([pc], [gc], [tc], weight_decay=0.0, momentum=momentum, lr=lr, dampening=0.0, nesterov=nesterov,
        maximize=False)
    L = (pc * torch.tensor(cP)).sum() + ((tc * torch.tensor(cT)).sum() if momentum > 0 else 0.0)
    dp, dg, dt = torch.autograd.grad(L, [p, g, t], allow_unused=True)
    o = oracle.sgd_bwd(cP, cT if momentum > 0 else None, lr, momentum, nesterov)
    assert np.allclose(o[0], dp.numpy(), rtol=1e-14, atol=0)
    assert _rel(o[1], dg.numpy()) < 1e-12
    if momentum > 0:
        assert _rel(o[2], dt.numpy()) < 1e-12


def test_sgd_vjp_central_differences():
    # the map is linear, so central differences are exact up to rounding
    n, lr, mu = 200, 0.05, 0.9
    p = normal(n, 0.05, "sgd", "p0", 3).astype(np.float64)
    g = normal(n, 0.01, "sgd", "grad", 3).astype(np.float64)
    t = normal(n, 0.01, "sgd", "mu", 3).astype(np.float64)
    cP = normal(n, 1.0, "sgd", "cot_p", 3).astype(np.float64)
    cT = normal(n, 1.0, "sgd", "cot_m", 3).astype(np.float64)
    for nest in (False, True):
        _, dg, dt = oracle.sgd_bwd(cP, cT, lr, mu, nest)
        h = 1e-3
        fp = oracle.sgd_fwd(p, g + h, t, lr, mu, nest)
        fm = oracle.sgd_fwd(p, g - h, t, lr, mu, nest)
        fd = (cP * (fp[0] - fm[0]) + cT * (fp[1] - fm[1])) / (2 * h)
        assert np.max(np.abs(fd - dg)) < 1e-9
        fp = oracle.sgd_fwd(p, g, t + h, lr, mu, nest)
        fm = oracle.sgd_fwd(p, g, t - h, lr, mu, nest)
        fd = (cP * (fp[0] - fm[0]) + cT * (fp[1] - fm[1])) / (2 * h)
        assert np.max(np.abs(fd - dt)) < 1e-9


# --------------------------------------------------------------- RMSProp

ALPHA, EPS = 0.99, 1e-8


@pytest.mark.parametrize("momentum", [0.0, 0.9])
def test_rmsprop_matches_torch_optim_over_steps(momentum):
    n, K, lr = 500, 15, 1e-3
    p0 = normal(n, 0.05, "rms", "p0").astype(np.float64)
    grads = [normal(n, 0.01, "rms", "grad", k).astype(np.float64) for k in range(K)]
    p, v, b = p0, np.zeros(n), None
    for g in grads:
        p, v, b1 = oracle.rmsprop_fwd(p, g, v, b, lr, ALPHA, EPS, 0.0, momentum)
        b = b1 if momentum > 0 else None
    tp = torch.tensor(p0, requires_grad=True)
    opt = torch.optim.RMSprop([tp], lr=lr, alpha=ALPHA, eps=EPS, momentum=momentum, centered=False)
    for g in grads:
        tp.grad = torch.tensor(g)
        opt.step()
    assert _rel(p - p0, tp.detach().numpy() - p0) < 1e-10
    assert _rel(v, opt.state[tp]["square_avg"].numpy()) < 1e-12


@pytest.mark.parametrize("eps_root", [0.0, 1e-8])
def test_rmsprop_step1_closed_form(eps_root):
    # from v = 0: v' = (1-alpha) g^2, u = -lr g / (sqrt((1-alpha) g^2 + eps_root) + eps)
    n, lr = 1000, 1e-3
    g = normal(n, 0.01, "rms", "grad", 7).astype(np.float64)
    p = normal(n, 0.05, "rms", "p0", 7).astype(np.float64)
    po, vo, _ = oracle.rmsprop_fwd(p, g, np.zeros(n), None, lr, ALPHA, EPS, eps_root, 0.0)
    assert _rel(vo, (1 - ALPHA) * g * g) < 1e-15
    assert _rel(po - p, -lr * g / (np.sqrt((1 - ALPHA) * g * g + eps_root) + EPS)) < 1e-9


@pytest.mark.parametrize("momentum", [0.0, 0.9])
def test_rmsprop_vjp_matches_torch_autograd(momentum):
    from torch.optim.rmsprop import rmsprop
    n, lr = 400, 1e-3
    p = torch.tensor(normal(n, 0.05, "rms", "p0", 8).astype(np.float64), requires_grad=True)
    g = torch.tensor(normal(n, 0.01, "rms", "grad", 8).astype(np.float64), requires_grad=True)
    v = torch.tensor(abs_normal(n, 1e-4, "rms", "nu", 8).astype(np.float64), requires_grad=True)
    b = torch.tensor(normal(n, 0.1, "rms", "mu", 8).astype(np.float64), requires_grad=True)
    cP, cV, cB = (normal(n, 1.0, "rms", t, 8).astype(np.float64) for t in ("cot_p", "cot_v", "cot_m"))
    pc, gc, vc, bc = p.clone(), g.clone(), v.clone(), b.clone()
    rmsprop([pc], [gc], [vc], [], [bc] if momentum > 0 else [], [torch.tensor(3.0, dtype=torch.float64)],
            foreach=False, differentiable=True, lr=lr, alpha=ALPHA, eps=EPS, weight_decay=0.0,
            momentum=momentum, centered=False)
    L = (pc * torch.tensor(cP)).sum() + (vc * torch.tensor(cV)).sum()
    if momentum > 0:
        L = L + (bc * torch.tensor(cB)).sum()
    dp, dg, dv, db = torch.autograd.grad(L, [p, g, v, b], allow_unused=True)
    o = oracle.rmsprop_bwd(cP, cV, cB if momentum > 0 else None, g.detach().numpy(), v.detach().numpy(), lr,
                           ALPHA, EPS, 0.0, momentum)
    mag = oracle.rmsprop_bwd_mag(cP, cV, cB if momentum > 0 else None, g.detach().numpy(), v.detach().numpy(),
                                 lr, ALPHA, EPS, 0.0, momentum)
    assert np.allclose(o[0], dp.numpy(), rtol=1e-14, atol=0)
    assert np.all(np.abs(o[1] - dg.numpy()) <= 1e-9 * mag[0])
    assert np.all(np.abs(o[2] - dv.numpy()) <= 1e-9 * mag[1])
    if momentum > 0:
        assert np.all(np.abs(o[3] - db.numpy()) <= 1e-12 * mag[2] + 1e-300)


@pytest.mark.parametrize("eps_root,momentum", [(0.0, 0.0), (1e-8, 0.0), (0.0, 0.9)])
def test_rmsprop_vjp_central_differences(eps_root, momentum):
    n, lr = 300, 1e-3
    p = normal(n, 0.05, "rms", "p0", 9).astype(np.float64)
    g = normal(n, 0.01, "rms", "grad", 9).astype(np.float64)
    v = abs_normal(n, 1e-4, "rms", "nu", 9).astype(np.float64) + 1e-7
    b = normal(n, 0.1, "rms", "mu", 9).astype(np.float64)
    cP, cV, cB = (normal(n, 1.0, "rms", t, 9).astype(np.float64) for t in ("cot_p", "cot_v", "cot_m"))
    cBm = cB if momentum > 0 else None
    _, dg, dv, db = oracle.rmsprop_bwd(cP, cV, cBm, g, v, lr, ALPHA, EPS, eps_root, momentum)
    mg = oracle.rmsprop_bwd_mag(cP, cV, cBm, g, v, lr, ALPHA, EPS, eps_root, momentum)

    def L(gg, vv, bb):
        po, vo, bo = oracle.rmsprop_fwd(p, gg, vv, bb, lr, ALPHA, EPS, eps_root, momentum)
        return cP * po + cV * vo + (cB * bo if momentum > 0 else 0.0)

    for which, (val, got, scale) in enumerate(((g, dg, mg[0]), (v, dv, mg[1]))):
        h = 1e-5 * np.maximum(np.abs(val), 1e-9)
        args_p = [g, v, b]
        args_m = [g, v, b]
        args_p[which] = val + h
        args_m[which] = val - h
        fd = (L(*args_p) - L(*args_m)) / (2 * h)
        assert np.max(np.abs(fd - got) / scale) < 1e-5, which
    if momentum > 0:
        h = 1e-4
        fd = (L(g, v, b + h) - L(g, v, b - h)) / (2 * h)
        assert np.max(np.abs(fd - db)) < 1e-9


def test_rmsprop_zero_over_zero_is_symmetric_derivative():
    # eps_root = 0, v = 0, g = 0: u(g) = -lr g / (sqrt(1-alpha) |g| + eps), whose
    # symmetric quotient is exactly -lr / (sqrt(1-alpha) h + eps) -> -lr / eps
    n, lr = 50, 1e-3
    cP = normal(n, 1.0, "rms", "cot_p", 10).astype(np.float64)
    z = np.zeros(n)
    _, dg, dv, _ = oracle.rmsprop_bwd(cP, None, None, z, z, lr, ALPHA, EPS, 0.0, 0.0)
    h = 1e-16
    up = oracle.rmsprop_fwd(z, z + h, z, None, lr, ALPHA, EPS, 0.0, 0.0)[0]
    um = oracle.rmsprop_fwd(z, z - h, z, None, lr, ALPHA, EPS, 0.0, 0.0)[0]
    assert _rel(dg, cP * (up - um) / (2 * h)) < 1e-6
    assert np.all(dv == 0.0)


def test_rmsprop_mag_bounds_values():
    n = 4000
    for momentum, eps_root, lr in ((0.0, 0.0, 1e-3), (0.9, 1e-8, 1e-3), (0.9, 1e-8, -1e-3)):
        p = normal(n, 0.05, "rmag", "p0").astype(np.float64)
        g = normal(n, 0.01, "rmag", "grad").astype(np.float64)
        v = abs_normal(n, 1e-4, "rmag", "nu").astype(np.float64)
        b = normal(n, 0.1, "rmag", "mu").astype(np.float64)
        cots = [normal(n, 1.0, "rmag", t).astype(np.float64) for t in ("cot_p", "cot_v", "cot_m")]
        f = oracle.rmsprop_fwd(p, g, v, b, lr, ALPHA, EPS, eps_root, momentum)
        fm = oracle.rmsprop_fwd_mag(p, g, v, b, lr, ALPHA, EPS, eps_root, momentum)
        for val, mg in zip(f, fm):
            assert np.all(np.abs(val) <= mg * (1 + 1e-12))
        bw = oracle.rmsprop_bwd(*cots, g, v, lr, ALPHA, EPS, eps_root, momentum)
        bm = oracle.rmsprop_bwd_mag(*cots, g, v, lr, ALPHA, EPS, eps_root, momentum)
        for val, mg in zip(bw[1:], bm):
            assert np.all(np.abs(val) <= mg * (1 + 1e-9))


def test_sgd_mag_bounds_values():
    # sums of |terms| bound |value| element by element (triangle inequality),
    # for either sign of the learning rate
    n = 4000
    for momentum, nesterov, lr in ((0.0, False, 0.1), (0.9, False, 0.05), (0.9, True, 0.05), (0.9, True, -0.05)):
        p = normal(n, 0.05, "smag", "p0").astype(np.float64)
        g = normal(n, 0.01, "smag", "grad").astype(np.float64)
        t = normal(n, 0.01, "smag", "mu").astype(np.float64)
        dP, dT = (normal(n, 1.0, "smag", tag).astype(np.float64) for tag in ("cot_p", "cot_m"))
        f = oracle.sgd_fwd(p, g, t, lr, momentum, nesterov)
        fm = oracle.sgd_fwd_mag(p, g, t, lr, momentum, nesterov)
        for val, mg in zip(f, fm):
            if momentum == 0.0 and mg is fm[1]:
                continue  # no trace without momentum
            assert np.all(np.abs(val) <= mg * (1 + 1e-12))
        bw = oracle.sgd_bwd(dP, dT, lr, momentum, nesterov)
        bm = oracle.sgd_bwd_mag(dP, dT, lr, momentum, nesterov)
        for val, mg in zip(bw[1:], bm):
            assert np.all(np.abs(val) <= mg * (1 + 1e-12))
