"""Pins of the oracle's K-step unrolled driver (Listing 1's loop, explicit
gradient): fp64 central differences of the K-step map, and autograd through
torch.optim's functional Adam in differentiable mode."""
import numpy as np
import pytest
import torch

import oracle
from workloads import HYPER, normal, abs_normal

LR, B1, B2, EPS = HYPER["lr"], HYPER["b1"], HYPER["b2"], HYPER["eps"]


def _inputs(n, K, seed, moments):
    p0 = normal(n, 0.05, "unr", "p0", seed).astype(np.float64)
    grads = np.stack([normal(n, 0.01, "unr", "grad", 100 * seed + k) for k in range(K)]).astype(np.float64)
    if moments:
        m0 = normal(n, 1e-3, "unr", "mu", seed).astype(np.float64)
        v0 = abs_normal(n, 1e-4, "unr", "nu", seed).astype(np.float64) + 1e-7
    else:
        m0 = np.zeros(n)
        v0 = np.zeros(n)
    cot = normal(n, 1.0, "unr", "cot_p", seed).astype(np.float64)
    return p0, grads, m0, v0, cot


@pytest.mark.parametrize("eps_root", [0.0, 1e-8])
@pytest.mark.parametrize("moments,count0", [(False, 0), (True, 100)])
def test_meta_gradient_central_differences(eps_root, moments, count0):
    # L = sum(cot * p_K).  With the gradients supplied from outside the K-step
    # map is elementwise, so one input family at a time is perturbed in all
    # coordinates at once (h_i ~ 1e-5 |x_i|), giving every partial from two runs.
    # Elements whose partial cancels to far below its family's typical size are
    # judged against 1% of that size (the quotient's rounding floor).
    n, K = 200, 5
    p0, grads, m0, v0, cot = _inputs(n, K, 1 + int(moments), moments)
    pK, mt, vt = oracle.unrolled_fwd(p0, grads, m0, v0, count0, LR, B1, B2, EPS, eps_root)
    dp0, dg, dm0, dv0 = oracle.unrolled_bwd(cot, grads, mt, vt, count0, LR, B1, B2, EPS, eps_root)

    def L(p0_, g_, m0_, v0_):
        return cot * oracle.unrolled_fwd(p0_, g_, m0_, v0_, count0, LR, B1, B2, EPS, eps_root)[0]

    def fd(which, k=None):
        args = [p0, grads.copy(), m0, v0]
        base = args[which] if k is None else args[1][k]
        rms = float(np.sqrt(np.mean(base * base))) or 1e-4
        h = 1e-5 * np.maximum(np.abs(base), 1e-2 * rms)
        plus = [a.copy() for a in args]
        minus = [a.copy() for a in args]
        if k is None:
            plus[which] = base + h
            minus[which] = base - h
        else:
            plus[1][k] = base + h
            minus[1][k] = base - h
        return (L(*plus) - L(*minus)) / (2 * h)

    def check(got, want, what):
        rms = float(np.sqrt(np.mean(want * want)))
        scale = np.maximum(np.abs(want), 1e-2 * rms)
        err = np.max(np.abs(got - want) / scale)
        assert err < 1e-5, (what, err)

    check(dp0, fd(0), "dp0")
    for k in range(K):
        check(dg[k], fd(1, k), "dg%d" % (k + 1))
    check(dm0, fd(2), "dm0")
    if moments:  # v0 = 0 sits on the boundary of the domain; only interior points
        check(dv0, fd(3), "dv0")


@pytest.mark.parametrize("count0", [0, 10])
def test_meta_gradient_matches_torch_autograd(count0):
    n, K = 300, 4
    p0, grads, m0, v0, cot = _inputs(n, K, 7, True)
    pK, mt, vt = oracle.unrolled_fwd(p0, grads, m0, v0, count0, LR, B1, B2, EPS, 0.0)
    dp0, dg, dm0, dv0 = oracle.unrolled_bwd(cot, grads, mt, vt, count0, LR, B1, B2, EPS, 0.0)

    from torch.optim.adam import adam
    leaves = [torch.tensor(x, requires_grad=True) for x in (p0, m0, v0)]
    gl = [torch.tensor(g, requires_grad=True) for g in grads]
    p, m, v = leaves[0].clone(), leaves[1].clone(), leaves[2].clone()
    for k in range(K):
        step = torch.tensor(float(count0 + k), dtype=torch.float64)
        adam([p], [gl[k].clone()], [m], [v], [], [step], foreach=False, capturable=False,
             differentiable=True, fused=None, grad_scale=None, found_inf=None,
             has_complex=False, amsgrad=False, beta1=B1, beta2=B2, lr=LR,
             weight_decay=0.0, eps=EPS, maximize=False)
    assert np.max(np.abs(p.detach().numpy() - pK)) < 1e-12
    out = torch.autograd.grad((p * torch.tensor(cot)).sum(), leaves + gl)
    ref = [o.numpy() for o in out]

    def close(a, b):
        scale = np.maximum(np.abs(b), 1e-3 * np.max(np.abs(b)))
        return np.max(np.abs(a - b) / scale) < 1e-8

    assert close(dp0, ref[0])
    assert close(dm0, ref[1])
    assert close(dv0, ref[2])
    for k in range(K):
        assert close(dg[k], ref[3 + k]), k


def test_trajectory_entry_zero_is_initial_state():
    n, K = 50, 3
    p0, grads, m0, v0, _ = _inputs(n, K, 3, True)
    pK, mt, vt = oracle.unrolled_fwd(p0, grads, m0, v0, 0, LR, B1, B2, EPS, 0.0)
    assert np.array_equal(mt[0], m0) and np.array_equal(vt[0], v0)
    # K = 1 is one plain step
    p1, m1, v1, _ = oracle.adam_fwd(p0, grads[0], m0, v0, 0, LR, B1, B2, EPS, 0.0)
    q1, mt1, vt1 = oracle.unrolled_fwd(p0, grads[:1], m0, v0, 0, LR, B1, B2, EPS, 0.0)
    assert np.array_equal(q1, p1) and np.array_equal(mt1[1], m1) and np.array_equal(vt1[1], v1)
