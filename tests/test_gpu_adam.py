"""GPU parity of the fused Adam forward and VJP kernels against the oracle.

Sizes span several workgroup tiles plus ragged tails (n % 4 != 0), the edge
cases n = 0..5, misaligned pointers (scalar path), in-place aliasing, and the
0/0 point of the VJP.  Tolerances: forward 1e-5, backward 1e-4, per element
relative to the oracle's term-magnitude scale (see tests/support.py).
"""
import numpy as np
import pytest
import torch

import oracle
from tests.support import BWD_RTOL, FWD_RTOL, assert_mag_close, assert_bits_equal
from workloads import HYPER, abs_normal, normal

pytestmark = pytest.mark.gpu

LR, B1, B2, EPS = HYPER["lr"], HYPER["b1"], HYPER["b2"], HYPER["eps"]

SIZES = [1, 2, 3, 4, 5, 7, 64, 1023, 1024, 4099, 256 * 4 * 4 * 3 + 5, 1_000_003]


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _host(t):
    return t.detach().cpu().numpy()


def _state(n, seed, moments, grad_std=0.01):
    p = normal(n, 0.05, "gpu", "p0", seed)
    g = normal(n, grad_std, "gpu", "grad", seed)
    if moments:
        m = normal(n, 1e-3, "gpu", "mu", seed)
        v = abs_normal(n, 1e-4, "gpu", "nu", seed)
    else:
        m = np.zeros(n, np.float32)
        v = np.zeros(n, np.float32)
    return p, g, m, v


def _run_fwd(p, g, m, v, count, eps_root, with_u=True):
    import paper_2211_06934_amd as P
    n = p.size
    tp, tg, tm, tv = map(_dev, (p, g, m, v))
    po, mo, vo = (torch.empty(n, dtype=torch.float32, device="cuda") for _ in range(3))
    uo = torch.empty(n, dtype=torch.float32, device="cuda") if with_u else None
    P.adam_fwd(tp, tg, tm, tv, count, LR, B1, B2, EPS, eps_root, po, mo, vo, uo)
    torch.cuda.synchronize()
    return [_host(x) for x in (po, mo, vo)] + ([_host(uo)] if with_u else [])


def _check_fwd(outs, p, g, m, v, count, eps_root):
    ref = oracle.adam_fwd(p, g, m, v, count, LR, B1, B2, EPS, eps_root)
    mag = oracle.adam_fwd_mag(p, g, m, v, count, LR, B1, B2, EPS, eps_root)
    for name, got, r, mg in zip(("p'", "m'", "v'", "u"), outs, ref, mag):
        assert_mag_close(got, r, mg, FWD_RTOL, name)


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("count,moments,eps_root", [(0, False, 0.0), (100, True, 0.0), (3, True, 1e-8)])
def test_adam_fwd_matches_oracle(n, count, moments, eps_root):
    p, g, m, v = _state(n, n % 97, moments)
    outs = _run_fwd(p, g, m, v, count, eps_root)
    _check_fwd(outs, p, g, m, v, count, eps_root)


def test_adam_fwd_without_update_output_and_n_zero():
    import paper_2211_06934_amd as P
    p, g, m, v = _state(4099, 5, True)
    outs = _run_fwd(p, g, m, v, 7, 0.0, with_u=False)
    ref = oracle.adam_fwd(p, g, m, v, 7, LR, B1, B2, EPS, 0.0)
    mag = oracle.adam_fwd_mag(p, g, m, v, 7, LR, B1, B2, EPS, 0.0)
    for got, r, mg in zip(outs, ref, mag):
        assert_mag_close(got, r, mg, FWD_RTOL)
    e = torch.empty(0, dtype=torch.float32, device="cuda")
    P.adam_fwd(e, e, e, e, 0, LR, B1, B2, EPS, 0.0, e, e, e)  # n == 0: no-op
    torch.cuda.synchronize()


def test_adam_fwd_in_place_aliasing():
    import paper_2211_06934_amd as P
    n = 100_003
    p, g, m, v = _state(n, 11, True)
    tp, tg, tm, tv = map(_dev, (p, g, m, v))
    P.adam_fwd(tp, tg, tm, tv, 5, LR, B1, B2, EPS, 1e-8, tp, tm, tv)
    torch.cuda.synchronize()
    _check_fwd([_host(tp), _host(tm), _host(tv)], p, g, m, v, 5, 1e-8)


@pytest.mark.parametrize("shift", [1, 2, 3])
def test_adam_fwd_misaligned_pointers_take_scalar_path(shift):
    import paper_2211_06934_amd as P
    n = 5000
    p, g, m, v = _state(n, 20 + shift, True)
    bufs = [torch.zeros(n + 4, dtype=torch.float32, device="cuda") for _ in range(7)]
    views = [b[shift:shift + n] for b in bufs]
    for vw, x in zip(views[:4], (p, g, m, v)):
        vw.copy_(_dev(x))
    P.adam_fwd(*views[:4], 9, LR, B1, B2, EPS, 0.0, *views[4:])
    torch.cuda.synchronize()
    _check_fwd([_host(x) for x in views[4:]], p, g, m, v, 9, 0.0)
    for b in bufs[4:]:  # nothing written outside the views
        hb = _host(b)
        assert np.all(hb[:shift] == 0) and np.all(hb[shift + n:] == 0)


def test_adam_fwd_step1_sign_update_exact_cases():
    # eps = eps_root = 0 at t = 1: u = -lr sign(g) (a closed form checked on GPU too)
    import paper_2211_06934_amd as P
    n = 4096 + 3
    g = normal(n, 0.01, "gpu", "grad", 31)
    g[g == 0] = 1e-3
    z = np.zeros(n, np.float32)
    tg = _dev(g)
    po, mo, vo, uo = (torch.empty(n, dtype=torch.float32, device="cuda") for _ in range(4))
    P.adam_fwd(_dev(z), tg, _dev(z), _dev(z), 0, LR, B1, B2, 0.0, 0.0, po, mo, vo, uo)
    u = _host(uo)
    assert np.all(np.abs(u + np.float32(LR) * np.sign(g)) <= 1e-6 * LR)


# ---------------------------------------------------------------- backward


def _run_bwd(cot, g, m, v, count, eps_root, with_mv, dparams_mode="none"):
    import paper_2211_06934_amd as P
    n = g.size
    tP = _dev(cot[0])
    tM = _dev(cot[1]) if with_mv else None
    tV = _dev(cot[2]) if with_mv else None
    dg, dm, dv = (torch.empty(n, dtype=torch.float32, device="cuda") for _ in range(3))
    if dparams_mode == "none":
        dp = None
    elif dparams_mode == "alias":
        dp = tP
    else:
        dp = torch.empty(n, dtype=torch.float32, device="cuda")
    P.adam_bwd(tP, tM, tV, _dev(g), _dev(m), _dev(v), count, LR, B1, B2, EPS, eps_root, dp, dg, dm, dv)
    torch.cuda.synchronize()
    return (None if dp is None else _host(dp)), _host(dg), _host(dm), _host(dv)


def _check_bwd(outs, cot, g, m, v, count, eps_root, with_mv):
    dM = cot[1] if with_mv else None
    dV = cot[2] if with_mv else None
    ref = oracle.adam_bwd(cot[0], dM, dV, g, m, v, count, LR, B1, B2, EPS, eps_root)
    mag = oracle.adam_bwd_mag(cot[0], dM, dV, g, m, v, count, LR, B1, B2, EPS, eps_root)
    if outs[0] is not None:
        assert_bits_equal(outs[0], cot[0], "dparams")
    for name, got, r, mg in zip(("dg", "dm", "dv"), outs[1:], ref[1:], mag):
        assert_mag_close(got, r, mg, BWD_RTOL, name)


def _cots(n, seed):
    return [normal(n, 1.0, "gpu", t, seed) for t in ("cot_p", "cot_m", "cot_v")]


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("count,moments,eps_root,with_mv",
                         [(0, False, 0.0, False), (0, False, 0.0, True), (100, True, 0.0, True),
                          (4, True, 1e-8, True), (2, True, 0.0, False)])
def test_adam_bwd_matches_oracle(n, count, moments, eps_root, with_mv):
    p, g, m, v = _state(n, 40 + n % 89, moments)
    cot = _cots(n, 40 + n % 89)
    outs = _run_bwd(cot, g, m, v, count, eps_root, with_mv)
    _check_bwd(outs, cot, g, m, v, count, eps_root, with_mv)


@pytest.mark.parametrize("mode", ["copy", "alias"])
def test_adam_bwd_dparams_is_identity(mode):
    n = 70_001
    p, g, m, v = _state(n, 50, True)
    cot = _cots(n, 50)
    outs = _run_bwd(cot, g, m, v, 6, 0.0, True, mode)
    _check_bwd(outs, cot, g, m, v, 6, 0.0, True)


def test_adam_bwd_zero_over_zero_points():
    # eps_root = 0 with v = 0 and g = 0 at scattered elements (fresh state): the
    # explicit 0/0 case must give the finite symmetric-derivative value.
    n = 10_000 + 1
    p, g, m, v = _state(n, 60, False)
    g[::7] = 0.0
    for count, mm in ((0, m), (5, normal(n, 1e-3, "gpu", "mu", 61))):
        mm = mm.copy()
        if count == 0:
            mm[:] = 0
        cot = _cots(n, 60)
        outs = _run_bwd(cot, g, mm, v, count, 0.0, True)
        assert all(np.all(np.isfinite(o)) for o in outs[1:])
        _check_bwd(outs, cot, g, mm, v, count, 0.0, True)


def test_adam_bwd_in_place_cotangents():
    import paper_2211_06934_amd as P
    n = 123_457
    p, g, m, v = _state(n, 70, True)
    cot = _cots(n, 70)
    tP, tM, tV = map(_dev, cot)
    dg = torch.empty(n, dtype=torch.float32, device="cuda")
    P.adam_bwd(tP, tM, tV, _dev(g), _dev(m), _dev(v), 12, LR, B1, B2, EPS, 0.0, None, dg, tM, tV)
    torch.cuda.synchronize()
    _check_bwd((None, _host(dg), _host(tM), _host(tV)), cot, g, m, v, 12, 0.0, True)


@pytest.mark.parametrize("shift", [1, 3])
def test_adam_bwd_misaligned(shift):
    import paper_2211_06934_amd as P
    n = 3001
    p, g, m, v = _state(n, 80 + shift, True)
    cot = _cots(n, 80 + shift)
    bufs = [torch.zeros(n + 4, dtype=torch.float32, device="cuda") for _ in range(9)]
    views = [b[shift:shift + n] for b in bufs]
    for vw, x in zip(views[:6], (*cot, g, m, v)):
        vw.copy_(_dev(x))
    P.adam_bwd(*views[:6], 3, LR, B1, B2, EPS, 1e-8, None, *views[6:])
    torch.cuda.synchronize()
    _check_bwd((None, *[_host(x) for x in views[6:]]), cot, g, m, v, 3, 1e-8, True)


def test_invalid_arguments_raise():
    import paper_2211_06934_amd as P
    t = torch.zeros(8, dtype=torch.float32, device="cuda")
    with pytest.raises(P.DiffoptError) as ei:
        P.adam_fwd(t, t, t, t, 0, LR, 1.0, B2, EPS, 0.0, t, t, t)
    assert ei.value.code == P.diffopt.DIFFOPT_EINVAL and "b1" in str(ei.value)
    with pytest.raises(P.DiffoptError):
        P.adam_fwd(t, t, t, t, -1, LR, B1, B2, EPS, 0.0, t, t, t)
    with pytest.raises(P.DiffoptError):
        P.adam_bwd(t, t, None, t, t, t, 0, LR, B1, B2, EPS, 0.0, None, t, t, t)
