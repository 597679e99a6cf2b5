"""Pins of the oracle's Adam forward and VJP against facts other than itself.

Each test ties one part of the oracle to a closed form, an invariant, a special
case that reduces to a library routine (torch.optim's Adam in fp64), or finite
differences.  A plausible slip in the oracle (a dropped term, wrong sign, wrong
bias-correction exponent, eps inside instead of outside the root, a transposed
operand) fails at least one of them.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import HYPER, normal, abs_normal

LR, B1, B2, EPS = HYPER["lr"], HYPER["b1"], HYPER["b2"], HYPER["eps"]


def _rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b) / np.maximum(np.abs(b), 1e-300)))


@pytest.mark.parametrize("eps_root", [0.0, 1e-8])
@pytest.mark.parametrize("eps", [1e-8, 0.0])
def test_step1_closed_form(eps_root, eps):
    # At t = 1 with zero moments the bias corrections undo the (1-b) factors:
    # m^ = g, v^ = g^2, so u = -lr g / (sqrt(g^2 + eps_root) + eps).
    g = normal(1000, 0.01, "pin", "grad").astype(np.float64)
    z = np.zeros_like(g)
    p = normal(1000, 0.05, "pin", "p0").astype(np.float64)
    p1, m1, v1, u = oracle.adam_fwd(p, g, z, z, 0, LR, B1, B2, eps, eps_root)
    expect_u = -LR * g / (np.sqrt(g * g + eps_root) + eps)
    assert _rel(u, expect_u) < 1e-14
    assert _rel(p1, p + expect_u) < 1e-14
    assert _rel(m1, (1 - B1) * g) < 1e-15
    assert _rel(v1, (1 - B2) * g * g) < 1e-15
    if eps == 0.0 and eps_root == 0.0:
        assert np.array_equal(np.sign(u), -np.sign(g))
        assert _rel(np.abs(u), np.full_like(u, LR)) < 1e-15


@pytest.mark.parametrize("eps_root", [0.0, 1e-8])
def test_constant_gradient_bias_correction(eps_root):
    # With a constant gradient and zero initial moments the bias-corrected
    # moments are exactly g and g^2 at every step, so the update never changes.
    g = normal(64, 0.01, "pin", "grad", 1).astype(np.float64)
    p = np.zeros_like(g)
    m = np.zeros_like(g)
    v = np.zeros_like(g)
    u_first = None
    for count in range(50):
        p, m, v, u = oracle.adam_fwd(p, g, m, v, count, LR, B1, B2, EPS, eps_root)
        if u_first is None:
            u_first = u
        assert _rel(u, u_first) < 1e-12, count


def test_zero_betas_reduce_to_normalised_gradient():
    # b1 = b2 = 0: m' = g, v' = g^2, c1 = c2 = 1 at any t; history is ignored.
    g = normal(256, 0.01, "pin", "grad", 2).astype(np.float64)
    m = normal(256, 1.0, "pin", "mu").astype(np.float64)
    v = abs_normal(256, 1.0, "pin", "nu").astype(np.float64)
    p = np.zeros_like(g)
    for eps_root in (0.0, 1e-6):
        _, m1, v1, u = oracle.adam_fwd(p, g, m, v, 7, LR, 0.0, 0.0, EPS, eps_root)
        assert _rel(u, -LR * g / (np.sqrt(g * g + eps_root) + EPS)) < 1e-14
        assert np.array_equal(m1, g)


def test_gradient_scale_invariance():
    # With eps = eps_root = 0, Adam's update is invariant to scaling the whole
    # gradient history by alpha > 0.
    n, K = 128, 6
    grads = np.stack([normal(n, 0.01, "pin", "grad", 10 + k) for k in range(K)]).astype(np.float64)
    p0 = normal(n, 0.05, "pin", "p0", 3).astype(np.float64)
    z = np.zeros(n)
    ref, _, _ = oracle.unrolled_fwd(p0, grads, z, z, 0, LR, B1, B2, 0.0, 0.0)
    for alpha in (1e3, 2.0 ** -10, 7.25):
        out, _, _ = oracle.unrolled_fwd(p0, alpha * grads, z, z, 0, LR, B1, B2, 0.0, 0.0)
        assert _rel(out - p0, ref - p0) < 1e-12


def test_update_sign_follows_first_moment():
    g = normal(512, 0.01, "pin", "grad", 4).astype(np.float64)
    m = normal(512, 0.01, "pin", "mu", 4).astype(np.float64)
    v = abs_normal(512, 1e-4, "pin", "nu", 4).astype(np.float64)
    _, m1, _, u = oracle.adam_fwd(np.zeros(512), g, m, v, 3, LR, B1, B2, EPS, 0.0)
    nz = m1 != 0
    assert np.array_equal(np.sign(u[nz]), -np.sign(m1[nz]))


def _torch_adam_steps(p0, grads, m0, v0, count0, lr, b1, b2, eps, differentiable=False):
    """torch.optim's functional single-tensor Adam in fp64 (library routine)."""
    from torch.optim.adam import adam
    p, m, v = p0, m0, v0
    for k, g in enumerate(grads):
        step = torch.tensor(float(count0 + k), dtype=torch.float64)
        adam([p], [g], [m], [v], [], [step], foreach=False, capturable=False,
             differentiable=differentiable, fused=None, grad_scale=None, found_inf=None,
             has_complex=False, amsgrad=False, beta1=b1, beta2=b2, lr=lr,
             weight_decay=0.0, eps=eps, maximize=False)
    return p, m, v


def test_matches_torch_optim_adam_fp64():
    # At eps_root = 0 the oracle must agree with torch.optim.Adam's single-tensor
    # path in fp64 (a different rounding order of the same textbook update).
    n, K = 1000, 20
    grads = np.stack([normal(n, 0.01, "pin", "grad", 30 + k) for k in range(K)]).astype(np.float64)
    p0 = normal(n, 0.05, "pin", "p0", 5).astype(np.float64)
    m0 = normal(n, 1e-3, "pin", "mu", 5).astype(np.float64)
    v0 = abs_normal(n, 1e-4, "pin", "nu", 5).astype(np.float64)
    for count0 in (0, 100):
        pk, mt, vt = oracle.unrolled_fwd(p0, grads, m0, v0, count0, LR, B1, B2, EPS, 0.0)
        tp, tm, tv = _torch_adam_steps(torch.tensor(p0), [torch.tensor(g) for g in grads],
                                       torch.tensor(m0), torch.tensor(v0), count0,
                                       LR, B1, B2, EPS)
        assert _rel(pk - p0, tp.numpy() - p0) < 1e-10
        # torch forms m' as a lerp, a different rounding order; the moments are
        # compared against their own scale
        assert np.max(np.abs(mt[-1] - tm.numpy())) < 1e-13 * np.max(np.abs(mt[-1]))
        assert np.max(np.abs(vt[-1] - tv.numpy())) < 1e-13 * np.max(np.abs(vt[-1]))


# ---------------------------------------------------------------- backward


@pytest.mark.parametrize("eps_root", [0.0, 1e-8])
def test_bwd_step1_closed_form(eps_root):
    # Zero moments, t = 1, zero moment cotangents:
    #   dg = -dP lr (eps_root + s eps) / (s d^2),  s = sqrt(g^2 + eps_root), d = s + eps
    #   dm = -b1 dP lr / ((1-b1) d)
    #   dv =  b2 dP lr g / (2 (1-b2) s d^2)
    n = 2000
    g = normal(n, 0.01, "pin", "grad", 6).astype(np.float64)
    dP = normal(n, 1.0, "pin", "cot_p", 6).astype(np.float64)
    z = np.zeros(n)
    dp, dg, dm, dv = oracle.adam_bwd(dP, None, None, g, z, z, 0, LR, B1, B2, EPS, eps_root)
    s = np.sqrt(g * g + eps_root)
    d = s + EPS
    assert np.array_equal(dp, dP)
    assert _rel(dg, -dP * LR * (eps_root + s * EPS) / (s * d * d)) < 1e-6
    assert _rel(dm, -B1 * dP * LR / ((1 - B1) * d)) < 1e-13
    assert _rel(dv, B2 * dP * LR * g / (2 * (1 - B2) * s * d * d)) < 1e-13


def test_bwd_step1_closed_form_dg_tight():
    # The plain chain rule cancels at t = 1 (relative error ~ ulp * g^2/(eps s)),
    # so the tight check uses a larger eps where the cancellation is mild.
    n = 500
    g = normal(n, 1.0, "pin", "grad", 7).astype(np.float64)
    dP = normal(n, 1.0, "pin", "cot_p", 7).astype(np.float64)
    z = np.zeros(n)
    eps, eps_root = 0.5, 0.25
    _, dg, _, _ = oracle.adam_bwd(dP, None, None, g, z, z, 0, LR, B1, B2, eps, eps_root)
    s = np.sqrt(g * g + eps_root)
    d = s + eps
    assert _rel(dg, -dP * LR * (eps_root + s * eps) / (s * d * d)) < 1e-12


def test_bwd_linear_in_cotangents():
    n = 300
    g = normal(n, 0.01, "pin", "grad", 8).astype(np.float64)
    m = normal(n, 1e-3, "pin", "mu", 8).astype(np.float64)
    v = abs_normal(n, 1e-4, "pin", "nu", 8).astype(np.float64)
    c1 = [normal(n, 1.0, "pin", t, 8).astype(np.float64) for t in ("cot_p", "cot_m", "cot_v")]
    c2 = [normal(n, 1.0, "pin", t, 9).astype(np.float64) for t in ("cot_p", "cot_m", "cot_v")]
    al, be = 0.75, -2.5
    r1 = oracle.adam_bwd(*c1, g, m, v, 4, LR, B1, B2, EPS, 1e-8)
    r2 = oracle.adam_bwd(*c2, g, m, v, 4, LR, B1, B2, EPS, 1e-8)
    r3 = oracle.adam_bwd(*[al * a + be * b for a, b in zip(c1, c2)], g, m, v, 4,
                         LR, B1, B2, EPS, 1e-8)
    for a, b, c in zip(r1, r2, r3):
        assert np.allclose(c, al * a + be * b, rtol=1e-12, atol=1e-300)


@pytest.mark.parametrize("count", [0, 100])
def test_bwd_matches_torch_autograd(count):
    # Autograd through torch.optim's functional Adam (differentiable mode) in
    # fp64 computes the same VJP by a route that shares nothing with the oracle.
    n = 400
    rng_p = normal(n, 0.05, "pin", "p0", 9).astype(np.float64)
    g = normal(n, 0.01, "pin", "grad", 9).astype(np.float64)
    m = normal(n, 1e-3, "pin", "mu", 9).astype(np.float64) if count else np.zeros(n)
    v = abs_normal(n, 1e-4, "pin", "nu", 9).astype(np.float64) if count else np.zeros(n)
    # avoid the s == 0 point, where the convention rather than calculus decides
    g[g == 0] = 1e-3
    cots = [normal(n, 1.0, "pin", t, 9).astype(np.float64) for t in ("cot_p", "cot_m", "cot_v")]
    leaves = [torch.tensor(x, requires_grad=True) for x in (rng_p, g, m, v)]
    tp, tm, tv = _torch_adam_steps(leaves[0].clone(), [leaves[1].clone()], leaves[2].clone(),
                                   leaves[3].clone(), count, LR, B1, B2, EPS, differentiable=True)
    L = (tp * torch.tensor(cots[0])).sum() + (tm * torch.tensor(cots[1])).sum() + \
        (tv * torch.tensor(cots[2])).sum()
    grads = torch.autograd.grad(L, leaves)
    dp, dg, dm, dv = oracle.adam_bwd(*cots, g, m, v, count, LR, B1, B2, EPS, 0.0)
    _, mag_dg, mag_dm, mag_dv = (None, *oracle.adam_bwd_mag(*cots, g, m, v, count, LR, B1, B2, EPS, 0.0))
    assert np.allclose(dp, grads[0].numpy(), rtol=1e-14, atol=0)
    assert np.all(np.abs(dg - grads[1].numpy()) <= 1e-7 * mag_dg)
    assert np.all(np.abs(dm - grads[2].numpy()) <= 1e-12 * mag_dm)
    assert np.all(np.abs(dv - grads[3].numpy()) <= 1e-9 * mag_dv)


def _fwd_outputs(x, count, eps_root):
    p, g, m, v = x
    p1, m1, v1, _ = oracle.adam_fwd(p, g, m, v, count, LR, B1, B2, EPS, eps_root)
    return p1, m1, v1


@pytest.mark.parametrize("eps_root", [0.0, 1e-8])
@pytest.mark.parametrize("count", [0, 5])
def test_bwd_central_differences(eps_root, count):
    # The forward is elementwise, so perturbing every coordinate of one input at
    # once by its own step h_i gives all n partials from two forward calls.
    n = 300
    p = normal(n, 0.05, "pin", "p0", 11).astype(np.float64)
    g = normal(n, 0.01, "pin", "grad", 11).astype(np.float64)
    m = normal(n, 1e-3, "pin", "mu", 11).astype(np.float64)
    v = abs_normal(n, 1e-4, "pin", "nu", 11).astype(np.float64) + 1e-6
    cots = [normal(n, 1.0, "pin", t, 11).astype(np.float64) for t in ("cot_p", "cot_m", "cot_v")]
    res = oracle.adam_bwd(*cots, g, m, v, count, LR, B1, B2, EPS, eps_root)
    mags = (np.abs(cots[0]), *oracle.adam_bwd_mag(*cots, g, m, v, count, LR, B1, B2, EPS, eps_root))
    base = [p, g, m, v]
    for which in range(4):
        h = 1e-6 * np.maximum(np.abs(base[which]), 1e-12)
        xp = list(base)
        xm = list(base)
        xp[which] = base[which] + h
        xm[which] = base[which] - h
        op = _fwd_outputs(xp, count, eps_root)
        om = _fwd_outputs(xm, count, eps_root)
        fd = sum(c * (a - b) for c, a, b in zip(cots, op, om)) / (2 * h)
        # relative to the sum of |terms|: a result that cancels to near zero is
        # judged on the scale of what cancelled
        err = np.abs(res[which] - fd) / mags[which]
        assert np.max(err) < 1e-5, (which, np.max(err))


def test_zero_over_zero_is_symmetric_derivative():
    # Reading of the 0/0 case: at eps_root = 0, v = 0, g = 0 the oracle's dg is
    # the limit of the symmetric difference quotient of the update in g.  Here
    # u(h) - u(-h) = -2 lr a h / (sqrt(b) h + eps) exactly, so the quotient tends
    # to -lr a / eps; m may be nonzero (then the one-sided slopes differ, by
    # ~1e9 here, so a loose bound on the rounding-limited quotient still decides).
    n = 64
    dP = normal(n, 1.0, "pin", "cot_p", 12).astype(np.float64)
    m = normal(n, 1e-3, "pin", "mu", 12).astype(np.float64)
    z = np.zeros(n)
    for count, mm, h, tol in ((0, z, 1e-15, 1e-6), (3, m, 1e-13, 1e-4)):
        _, dg, dm, dv = oracle.adam_bwd(dP, None, None, z, mm, z, count, LR, B1, B2, EPS, 0.0)
        assert np.all(np.isfinite(dg)) and np.all(np.isfinite(dv))
        up = oracle.adam_fwd(z, z + h, mm, z, count, LR, B1, B2, EPS, 0.0)[0]
        um = oracle.adam_fwd(z, z - h, mm, z, count, LR, B1, B2, EPS, 0.0)[0]
        fd = dP * (up - um) / (2 * h)
        assert _rel(dg, fd) < tol, count
        assert np.all(dv == 0.0)
    # The nu-cotangent there.  From a fresh state (m = 0, the case the inner
    # loop reaches), m' = 0, so the update is 0 for every v >= 0 and the exact
    # derivative in v is 0: the one-sided difference quotient pins the value.
    # With m != 0 the one-sided slope is unbounded, and 0 is a convention.
    _, _, _, dv = oracle.adam_bwd(dP, None, None, z, z, z, 0, LR, B1, B2, EPS, 0.0)
    for h in (1e-30, 1e-12, 1e-4):
        u1 = oracle.adam_fwd(z, z, z, z + h, 0, LR, B1, B2, EPS, 0.0)[0]
        u0 = oracle.adam_fwd(z, z, z, z, 0, LR, B1, B2, EPS, 0.0)[0]
        assert np.array_equal(dv, dP * (u1 - u0) / h)


def test_mag_bounds_values():
    # The tolerance scales are sums of |terms|, so they bound |value| for every
    # element (triangle inequality); a dropped term usually breaks this.
    n = 5000
    for count, eps_root, lr in ((0, 0.0, LR), (7, 1e-8, LR), (100, 0.0, LR), (7, 1e-8, -LR)):
        p = normal(n, 0.05, "mag", "p0", count).astype(np.float64)
        g = normal(n, 0.01, "mag", "grad", count).astype(np.float64)
        m = normal(n, 1e-3, "mag", "mu", count).astype(np.float64) if count else np.zeros(n)
        v = abs_normal(n, 1e-4, "mag", "nu", count).astype(np.float64) if count else np.zeros(n)
        cots = [normal(n, 1.0, "mag", t, count).astype(np.float64) for t in ("cot_p", "cot_m", "cot_v")]
        f = oracle.adam_fwd(p, g, m, v, count, lr, B1, B2, EPS, eps_root)
        fm = oracle.adam_fwd_mag(p, g, m, v, count, lr, B1, B2, EPS, eps_root)
        for val, mg in zip(f, fm):
            assert np.all(np.abs(val) <= mg * (1 + 1e-12))
        b = oracle.adam_bwd(*cots, g, m, v, count, lr, B1, B2, EPS, eps_root)
        bm = oracle.adam_bwd_mag(*cots, g, m, v, count, lr, B1, B2, EPS, eps_root)
        for val, mg in zip(b[1:], bm):
            assert np.all(np.abs(val) <= mg * (1 + 1e-9))
