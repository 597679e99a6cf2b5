"""Hyper-parameters away from the defaults, through the single-step kernels
and the fused K-step driver, against the oracle.  The coefficients (1-b1,
1-b2, 1/c1, 1/c2, lr/c1, ...) are derived on the host in fp64 and rounded once
to fp32, so every combination must meet the same per-element bars (1e-5
forward, 1e-4 backward of the term scale): b1 = b2 = 0 (no averaging),
heavy averaging (b2 = 0.9999), large eps and eps_root, eps = 0 with
eps_root > 0, a negative learning rate (ascent), lr = 0, and a late step
(count 10^6, bias corrections ~ 1).  SGD (either sign of lr, momentum up to
0.99, Nesterov, lr = 0) and RMSProp (alpha = 0, heavy averaging, eps = 0 with
eps_root > 0, lr < 0, with and without momentum) the same way."""
import numpy as np
import pytest
import torch

import oracle
from tests.support import BWD_RTOL, FWD_RTOL, assert_mag_close

pytestmark = pytest.mark.gpu

HYPERS = [  # lr, b1, b2, eps, eps_root, count
    (0.1, 0.0, 0.0, 1e-8, 0.0, 0),
    (1e-3, 0.5, 0.9, 1e-3, 1e-6, 3),
    (1e-2, 0.99, 0.9999, 1e-8, 1e-12, 0),
    (1e-3, 0.9, 0.999, 0.0, 1e-8, 2),
    (-1e-3, 0.9, 0.999, 1e-8, 0.0, 5),
    (0.0, 0.9, 0.999, 1e-8, 0.0, 1),
    (3e-4, 0.9, 0.999, 1e-8, 0.0, 10 ** 6),
]


def _inputs(n, seed):
    rng = np.random.default_rng(seed)
    f = lambda x: x.astype(np.float32)  # noqa: E731
    return (f(rng.standard_normal(n) * 0.05), f(rng.standard_normal(n) * 1e-2), f(rng.standard_normal(n) * 1e-3),
            f(np.abs(rng.standard_normal(n)) * 1e-4), f(rng.standard_normal(n)), f(rng.standard_normal(n)),
            f(rng.standard_normal(n)))


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _h(t):
    return t.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("hyper", HYPERS, ids=lambda h: "lr%g-b1%g-b2%g-eps%g-er%g-c%d" % h)
def test_single_step(hyper):
    import paper_2211_06934_amd as P
    lr, b1, b2, eps, er, count = hyper
    n = 2 * 4096 + 7
    p, g, m, v, dP, dM, dV = _inputs(n, 1)
    po, mo, vo, dg, dm, dv = (torch.empty(n, device="cuda") for _ in range(6))
    P.adam_fwd(_dev(p), _dev(g), _dev(m), _dev(v), count, lr, b1, b2, eps, er, po, mo, vo)
    P.adam_bwd(_dev(dP), _dev(dM), _dev(dV), _dev(g), _dev(m), _dev(v), count, lr, b1, b2, eps, er, None, dg, dm, dv)
    torch.cuda.synchronize()
    ref = oracle.adam_fwd(p, g, m, v, count, lr, b1, b2, eps, er)
    mag = oracle.adam_fwd_mag(p, g, m, v, count, lr, b1, b2, eps, er)
    for got, r, mg, what in zip((po, mo, vo), ref[:3], mag[:3], ("p'", "m'", "v'")):
        assert_mag_close(_h(got), r, mg, FWD_RTOL, what)
    ref = oracle.adam_bwd(dP, dM, dV, g, m, v, count, lr, b1, b2, eps, er)
    mag = oracle.adam_bwd_mag(dP, dM, dV, g, m, v, count, lr, b1, b2, eps, er)
    for got, r, mg, what in zip((dg, dm, dv), ref[1:], mag, ("dg", "dm", "dv")):
        assert_mag_close(_h(got), r, mg, BWD_RTOL, what)


@pytest.mark.parametrize("hyper", HYPERS, ids=lambda h: "lr%g-b1%g-b2%g-eps%g-er%g-c%d" % h)
def test_fused_driver(hyper):
    # K = 4 from a warm state: the whole trajectory stored (checked step by
    # step against the oracle) and recomputed (bit for bit the same)
    import paper_2211_06934_amd as P
    lr, b1, b2, eps, er, count = hyper
    K, n = 4, 4096 + 3
    p, _, m0, v0, cot, _, _ = _inputs(n, 2)
    gs = [_inputs(n, 10 + k)[1] for k in range(K)]
    gd = [_dev(x) for x in gs]
    runs = []
    for stored in (True, False):
        mt = [_dev(m0)] + [torch.empty(n, device="cuda") if stored or k == K else None for k in range(1, K + 1)]
        vt = [_dev(v0)] + [torch.empty(n, device="cuda") if stored or k == K else None for k in range(1, K + 1)]
        pK = torch.empty(n, device="cuda")
        dg = [torch.empty(n, device="cuda") for _ in range(K)]
        dm0, dv0 = torch.empty(n, device="cuda"), torch.empty(n, device="cuda")
        P.adam_unrolled_fwd(_dev(p), gd, mt, vt, pK, count, lr, b1, b2, eps, er)
        P.adam_unrolled_bwd(_dev(cot), gd, mt, vt, dg, dm0, dv0, count, lr, b1, b2, eps, er)
        runs.append((pK, mt, vt, dg, dm0, dv0))
    torch.cuda.synchronize()
    a, b = runs
    for x, y in zip([a[0], *a[3], a[4], a[5], a[1][K], a[2][K]], [b[0], *b[3], b[4], b[5], b[1][K], b[2][K]]):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))
    pK, mt, vt, dg, dm0, dv0 = a
    G = np.stack([x.astype(np.float64) for x in gs])
    hm, hv = np.stack([_h(x) for x in mt]), np.stack([_h(x) for x in vt])
    for k in range(1, K + 1):
        ref = oracle.adam_fwd(p, G[k - 1], hm[k - 1], hv[k - 1], count + k - 1, lr, b1, b2, eps, er)
        mag = oracle.adam_fwd_mag(p, G[k - 1], hm[k - 1], hv[k - 1], count + k - 1, lr, b1, b2, eps, er)
        assert_mag_close(hm[k], ref[1], mag[1], FWD_RTOL, "m_%d" % k)
        assert_mag_close(hv[k], ref[2], mag[2], FWD_RTOL, "v_%d" % k)
    hc = cot.astype(np.float64)
    _, dg_l, dm0_l, dv0_l = oracle.unrolled_bwd(hc, G, hm, hv, count, lr, b1, b2, eps, er)
    magM, magV = np.zeros(n), np.zeros(n)
    for k in range(K, 0, -1):
        mg, mm, mv = oracle.adam_bwd_mag(hc, magM, magV, G[k - 1], hm[k - 1], hv[k - 1], count + k - 1, lr, b1, b2,
                                         eps, er)
        assert_mag_close(_h(dg[k - 1]), dg_l[k - 1], mg, BWD_RTOL, "dg_%d" % k)
        magM, magV = mm, mv
    assert_mag_close(_h(dm0), dm0_l, magM, BWD_RTOL, "dmu0")
    assert_mag_close(_h(dv0), dv0_l, magV, BWD_RTOL, "dnu0")


SGD_HYPERS = [(0.1, 0.0, False), (-0.05, 0.9, True), (0.01, 0.99, False), (0.0, 0.9, True)]
RMS_HYPERS = [  # lr, alpha, eps, eps_root, momentum
    (1e-3, 0.0, 1e-8, 0.0, 0.0),
    (1e-2, 0.5, 1e-3, 1e-6, 0.9),
    (-1e-3, 0.99, 0.0, 1e-8, 0.0),
    (1e-3, 0.999, 1e-8, 0.0, 0.99),
]


@pytest.mark.parametrize("hyper", SGD_HYPERS, ids=lambda h: "lr%g-mom%g-nest%d" % h)
def test_sgd_hyper(hyper):
    import paper_2211_06934_amd as P
    lr, mom, nest = hyper
    n = 4096 + 9
    p, g, t, _, dP, dT, _ = _inputs(n, 3)
    po, to, dg, dt = (torch.empty(n, device="cuda") for _ in range(4))
    P.sgd_fwd(_dev(p), _dev(g), _dev(t), lr, mom, nest, po, to if mom > 0 else None)
    P.sgd_bwd(_dev(dP), _dev(dT) if mom > 0 else None, lr, mom, nest, dg, dt if mom > 0 else None)
    torch.cuda.synchronize()
    ref, mag = oracle.sgd_fwd(p, g, t, lr, mom, nest), oracle.sgd_fwd_mag(p, g, t, lr, mom, nest)
    assert_mag_close(_h(po), ref[0], mag[0], FWD_RTOL, "p'")
    if mom > 0:
        assert_mag_close(_h(to), ref[1], mag[1], FWD_RTOL, "t'")
    ref = oracle.sgd_bwd(dP, dT if mom > 0 else None, lr, mom, nest)
    mag = oracle.sgd_bwd_mag(dP, dT if mom > 0 else None, lr, mom, nest)
    assert_mag_close(_h(dg), ref[1], mag[0], BWD_RTOL, "dg")
    if mom > 0:
        assert_mag_close(_h(dt), ref[2], mag[1], BWD_RTOL, "dt")


@pytest.mark.parametrize("hyper", RMS_HYPERS, ids=lambda h: "lr%g-a%g-eps%g-er%g-mom%g" % h)
def test_rmsprop_hyper(hyper):
    import paper_2211_06934_amd as P
    lr, alpha, eps, er, mom = hyper
    n = 4096 + 9
    p, g, b, v, dP, dV, dB = _inputs(n, 4)
    po, vo, bo, dg, dv, db = (torch.empty(n, device="cuda") for _ in range(6))
    m = mom > 0
    P.rmsprop_fwd(_dev(p), _dev(g), _dev(v), _dev(b) if m else None, lr, alpha, eps, er, mom, po, vo,
                  bo if m else None)
    P.rmsprop_bwd(_dev(dP), _dev(dV), _dev(dB) if m else None, _dev(g), _dev(v), lr, alpha, eps, er, mom, dg, dv,
                  db if m else None)
    torch.cuda.synchronize()
    bb = b if m else None
    ref = oracle.rmsprop_fwd(p, g, v, bb, lr, alpha, eps, er, mom)
    mag = oracle.rmsprop_fwd_mag(p, g, v, bb, lr, alpha, eps, er, mom)
    outs = (po, vo, bo) if m else (po, vo)
    for got, r, mg, what in zip(outs, ref, mag, ("p'", "v'", "b'")):
        assert_mag_close(_h(got), r, mg, FWD_RTOL, what)
    ref = oracle.rmsprop_bwd(dP, dV, dB if m else None, g, v, lr, alpha, eps, er, mom)[1:]
    mag = oracle.rmsprop_bwd_mag(dP, dV, dB if m else None, g, v, lr, alpha, eps, er, mom)
    outs = (dg, dv, db) if m else (dg, dv)
    for got, r, mg, what in zip(outs, ref, mag, ("dg", "dv", "db")):
        assert_mag_close(_h(got), r, mg, BWD_RTOL, what)
