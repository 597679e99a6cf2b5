"""Tiny denominators in the VJPs.  With eps = 0 (allowed) and tiny gradients,
s d^2 of the Adam VJP (and of RMSProp's) underflows in fp32 while the
quotients it divides are finite: with a fresh state and eps = eps_root = 0 the
dupdate coefficient of dg is exactly 0 and the nu-cotangent is large but
representable.  The kernels must return those values (a reciprocal of the
underflowed product gives inf, and 0 * inf NaN), through every path that
runs the step: the single-step kernels, the fused K-step driver with the
trajectory recomputed, the leaf-direct step, and RMSProp flat and
leaf-direct.  Checked against the oracle element by element (1e-5 / 1e-4 of
the term scale), except for dg of a single step from a fresh state with
eps = eps_root = 0: there the update is -lr (1-b1)/(c1 sqrt(b)) sign(g)
(RMSProp: -lr sign(g)/sqrt(1-alpha)), constant in g, so the closed form fixes
the dupdate part of dg at exactly 0, while the oracle's plain chain rule
subtracts two terms of size lr a / s and keeps their fp64 rounding
difference (about 1e-16 lr a / s, far above 0)."""
import numpy as np
import pytest
import torch

import oracle
from tests.support import BWD_RTOL, FWD_RTOL, assert_mag_close
from workloads import HYPER

pytestmark = pytest.mark.gpu

LR, B1, B2 = HYPER["lr"], HYPER["b1"], HYPER["b2"]


def _tiny(n, seed, lo=-14.0, hi=-12.0):
    rng = np.random.default_rng(seed)
    return (np.where(rng.random(n) < 0.5, -1.0, 1.0) * 10.0 ** rng.uniform(lo, hi, n)).astype(np.float32)


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def _h(t):
    return t.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("eps,eps_root", [(0.0, 0.0), (0.0, 1e-30), (1e-8, 0.0)])
def test_adam_single_step(eps, eps_root):
    import paper_2211_06934_amd as P
    n = 3 * 4096 + 5
    rng = np.random.default_rng(3)
    g = _tiny(n, 1)
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    z = np.zeros(n, np.float32)
    dP = rng.standard_normal(n).astype(np.float32)
    po, mo, vo, dg, dm, dv = (torch.empty(n, device="cuda") for _ in range(6))
    P.adam_fwd(_dev(p), _dev(g), _dev(z), _dev(z), 0, LR, B1, B2, eps, eps_root, po, mo, vo)
    P.adam_bwd(_dev(dP), None, None, _dev(g), _dev(z), _dev(z), 0, LR, B1, B2, eps, eps_root, None, dg, dm, dv)
    torch.cuda.synchronize()
    ref = oracle.adam_fwd(p, g, z, z, 0, LR, B1, B2, eps, eps_root)
    mag = oracle.adam_fwd_mag(p, g, z, z, 0, LR, B1, B2, eps, eps_root)
    for got, r, m, what in zip((po, mo, vo), ref[:3], mag[:3], ("p'", "m'", "v'")):
        assert_mag_close(_h(got), r, m, FWD_RTOL, what)
    zz = np.zeros(n)
    ref = oracle.adam_bwd(dP, zz, zz, g, z, z, 0, LR, B1, B2, eps, eps_root)
    mag = oracle.adam_bwd_mag(dP, zz, zz, g, z, z, 0, LR, B1, B2, eps, eps_root)
    for got, r, m, what in zip((dg, dm, dv), ref[1:], mag, ("dg", "dm", "dv")):
        assert torch.isfinite(got).all(), what
        if what == "dg" and eps == 0.0 and eps_root == 0.0:
            assert np.all(_h(got) == 0.0), "dg: the closed form is 0"
            continue
        assert_mag_close(_h(got), r, m, BWD_RTOL, what)


def test_adam_fused_driver_and_leaf_direct():
    # eps = eps_root = 0, fresh state, K = 3: the fused driver (whole
    # trajectory stored, then recomputed: both runs must agree bit for bit)
    # against the oracle's backward on the GPU's own trajectory, and the
    # leaf-direct single step against the oracle
    import paper_2211_06934_amd as P
    K, numel = 3, [4096 + 3, 0, 2 * 4096 + 1]
    n = sum(numel)
    rng = np.random.default_rng(5)
    p = (rng.standard_normal(n) * 0.05).astype(np.float32)
    gs = [_tiny(n, 10 + k) for k in range(K)]
    cot = rng.standard_normal(n).astype(np.float32)
    e = lambda: torch.empty(n, device="cuda")  # noqa: E731
    gd = [_dev(x) for x in gs]
    runs = []
    for stored in (True, False):
        mt = [torch.zeros(n, device="cuda")] + [e() if stored or k == K else None for k in range(1, K + 1)]
        vt = [torch.zeros(n, device="cuda")] + [e() if stored or k == K else None for k in range(1, K + 1)]
        pK, dg, dm0, dv0 = e(), [e() for _ in range(K)], e(), e()
        P.adam_unrolled_fwd(_dev(p), gd, mt, vt, pK, 0, LR, B1, B2, 0.0, 0.0)
        P.adam_unrolled_bwd(_dev(cot), gd, mt, vt, dg, dm0, dv0, 0, LR, B1, B2, 0.0, 0.0)
        runs.append((mt, vt, dg, dm0, dv0))
    torch.cuda.synchronize()
    for a, b in zip(runs[0][2] + [runs[0][3], runs[0][4]], runs[1][2] + [runs[1][3], runs[1][4]]):
        assert torch.isfinite(a).all()
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    mt, vt, dg, dm0, dv0 = runs[0]
    G = np.stack([x.astype(np.float64) for x in gs])
    hm, hv = np.stack([_h(x) for x in mt]), np.stack([_h(x) for x in vt])
    hc = cot.astype(np.float64)
    _, dg_l, dm0_l, dv0_l = oracle.unrolled_bwd(hc, G, hm, hv, 0, LR, B1, B2, 0.0, 0.0)
    magM, magV = np.zeros(n), np.zeros(n)
    for k in range(K, 0, -1):
        mg, mm, mv = oracle.adam_bwd_mag(hc, magM, magV, G[k - 1], hm[k - 1], hv[k - 1], k - 1, LR, B1, B2, 0.0, 0.0)
        assert_mag_close(_h(dg[k - 1]), dg_l[k - 1], mg, BWD_RTOL, "dg_%d" % k)
        magM, magV = mm, mv
    assert_mag_close(_h(dm0), dm0_l, magM, BWD_RTOL, "dmu0")
    assert_mag_close(_h(dv0), dv0_l, magV, BWD_RTOL, "dnu0")

    table = P.segtable_create(numel)
    split = lambda x: [t.contiguous() for t in torch.split(_dev(x), numel)]  # noqa: E731
    ptr = lambda ls: torch.tensor([t.data_ptr() for t in ls], dtype=torch.int64, device="cuda")  # noqa: E731
    lp, lg, lz, lc = split(p), split(gs[0]), split(np.zeros(n)), split(cot)
    lpo, lmo, lvo, ldg, ldm, ldv = ([torch.empty(k, device="cuda") for k in numel] for _ in range(6))
    P.adam_fwd_tree(table, ptr(lp), ptr(lg), ptr(lz), ptr(lz), 0, LR, B1, B2, 0.0, 0.0, ptr(lpo), ptr(lmo),
                    ptr(lvo))
    P.adam_bwd_tree(table, ptr(lc), None, None, ptr(lg), ptr(lz), ptr(lz), 0, LR, B1, B2, 0.0, 0.0, ptr(ldg),
                    ptr(ldm), ptr(ldv))
    torch.cuda.synchronize()
    zz = np.zeros(n)
    ref = oracle.adam_bwd(cot, zz, zz, gs[0], zz, zz, 0, LR, B1, B2, 0.0, 0.0)
    mag = oracle.adam_bwd_mag(cot, zz, zz, gs[0], zz, zz, 0, LR, B1, B2, 0.0, 0.0)
    for got, r, m, what in zip((ldg, ldm, ldv), ref[1:], mag, ("dg", "dm", "dv")):
        got = torch.cat(got)
        assert torch.isfinite(got).all(), what
        if what == "dg":
            assert np.all(_h(got) == 0.0), "dg: the closed form is 0"
            continue
        assert_mag_close(_h(got), r, m, BWD_RTOL, what)


def test_rmsprop_flat_and_leaf_direct():
    import paper_2211_06934_amd as P
    numel = [4096 + 3, 5, 2 * 4096 + 1]
    n = sum(numel)
    rng = np.random.default_rng(7)
    g = _tiny(n, 2, -16.0, -13.0)
    v = np.zeros(n, np.float32)
    dP, dV = (rng.standard_normal(n).astype(np.float32) for _ in range(2))
    hp = (1e-3, 0.99, 0.0, 0.0, 0.0)  # lr, alpha, eps, eps_root, momentum
    dg, dv = torch.empty(n, device="cuda"), torch.empty(n, device="cuda")
    P.rmsprop_bwd(_dev(dP), _dev(dV), None, _dev(g), _dev(v), *hp, dg, dv)
    table = P.segtable_create(numel)
    split = lambda x: [t.contiguous() for t in torch.split(_dev(x), numel)]  # noqa: E731
    ptr = lambda ls: torch.tensor([t.data_ptr() for t in ls], dtype=torch.int64, device="cuda")  # noqa: E731
    ldg, ldv = ([torch.empty(k, device="cuda") for k in numel] for _ in range(2))
    ins = [split(x) for x in (dP, dV, g, v)]  # held until the kernel has run
    P.rmsprop_bwd_tree(table, ptr(ins[0]), ptr(ins[1]), None, ptr(ins[2]), ptr(ins[3]), *hp, ptr(ldg), ptr(ldv))
    torch.cuda.synchronize()
    ref = oracle.rmsprop_bwd(dP, dV, None, g, v, *hp)[1:3]
    mag = oracle.rmsprop_bwd_mag(dP, dV, None, g, v, *hp)[:2]
    # dg: the update's part vanishes (closed form), leaving the nu path
    # 2 (1 - alpha) g dV, whose fp32 product is within one rounding per factor
    dg_exact = 2.0 * (1.0 - hp[1]) * g.astype(np.float64) * dV.astype(np.float64)
    for got, what in ((dg, "dg"), (torch.cat(ldg), "tree dg")):
        assert torch.isfinite(got).all(), what
        assert np.all(np.abs(_h(got) - dg_exact) <= 1e-6 * np.abs(dg_exact)), what
    for got, what in ((dv, "dv"), (torch.cat(ldv), "tree dv")):
        assert torch.isfinite(got).all(), what
        assert_mag_close(_h(got), ref[1], mag[1], BWD_RTOL, what)
