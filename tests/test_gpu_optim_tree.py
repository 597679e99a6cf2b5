"""GPU parity of the leaf-direct ("tree map") SGD-momentum and RMSProp steps
and VJPs, and of MetaSGD / MetaRMSProp inside a MAML inner loop.

The tree-map step is by definition flatten -> flat step -> unflatten, so the
expected values are the oracle's flat step on the packed leaves (forward 1e-5,
backward 1e-4 of the term-magnitude scale), and the GPU's tree result must
also equal the GPU's flat kernels on the flattened tree bit for bit (the same
per-element arithmetic).  Trees hold empty and tiny leaves, separate
allocations and views out of 16-byte phase (element path); a small tree
(9 nonempty leaves) takes the one-element-per-lane small-tree kernel.  The MAML tests
take the meta-gradient through K inner steps of the conv-net, against the same
loop built on torch.optim's functional SGD / RMSprop, in fp64 on the CPU and in
fp32 on the GPU.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from tests.support import BWD_RTOL, FWD_RTOL, assert_mag_close
from tests.test_gpu_maml import ConvNet, _normrel, _task, torch32_spread
from tests.test_gpu_treemap import _device_tree, _empty_like_tree, _ptrs, _split
from workloads import abs_normal, normal, random_shapes

pytestmark = pytest.mark.gpu

ALPHA, EPS = 0.99, 1e-8


def _numel(seed, size="many"):
    """"many": 84 nonempty leaves (the tiled kernels); "small": 9 nonempty
    leaves and 7,377 elements (the small-tree kernels, one element per lane)."""
    if size == "small":
        return [0, 3, 40, 1600, 1, 0, 4096, 777, 5, 855, 0]
    shapes = random_shapes(80, 3000, seed=seed)
    numel = [int(np.prod(s)) for s in shapes]
    return [0, 3] + numel[:40] + [0, 1, 4096, 5] + numel[40:]


def _flat(tree):
    return torch.cat([x.reshape(-1) for x in tree]).cpu().numpy() if tree else np.zeros(0, np.float32)


def _bits(tree):
    return torch.cat([x.reshape(-1) for x in tree]).view(torch.int32).cpu().numpy()


@pytest.mark.parametrize("size", ["many", "small"])
@pytest.mark.parametrize("mode", ["separate", "packed-views"])
@pytest.mark.parametrize("momentum,with_trace,nesterov,with_dt", [
    (0.0, False, False, False), (0.9, False, False, False), (0.9, True, False, True), (0.9, True, True, True),
    (0.9, False, True, False)])
def test_sgd_tree_matches_oracle_and_flat(mode, momentum, with_trace, nesterov, with_dt, size):
    import paper_2211_06934_amd as P
    numel = _numel(3, size)
    n = sum(numel)
    table = P.segtable_create(numel)
    lr = 0.05
    hp, hg, ht = normal(n, 0.05, "st", "p0", 1), normal(n, 0.01, "st", "grad", 1), normal(n, 0.01, "st", "mu", 1)
    hP, hT = normal(n, 1.0, "st", "cot_p", 1), normal(n, 1.0, "st", "cot_m", 1)
    tree = lambda a, s: _device_tree(_split(a, numel), mode, s)  # noqa: E731
    p, g, P_ = tree(hp, 1), tree(hg, 2), tree(hP, 4)
    t = tree(ht, 3) if with_trace else None
    T = tree(hT, 5) if with_dt else None
    mom = momentum > 0
    po = _empty_like_tree(p, mode, 6)
    to = _empty_like_tree(p, mode, 7) if mom else None
    dg = _empty_like_tree(p, mode, 8)
    dt = _empty_like_tree(p, mode, 9) if mom else None
    pp = lambda x: None if x is None else _ptrs(x)  # noqa: E731
    P.sgd_fwd_tree(table, pp(p), pp(g), pp(t), lr, momentum, nesterov, pp(po), pp(to))
    P.sgd_bwd_tree(table, pp(P_), pp(T), lr, momentum, nesterov, pp(dg), pp(dt))
    torch.cuda.synchronize()
    rp, rt = oracle.sgd_fwd(hp, hg, ht if with_trace else None, lr, momentum, nesterov)
    mp, mt = oracle.sgd_fwd_mag(hp, hg, ht if with_trace else None, lr, momentum, nesterov)
    assert_mag_close(_flat(po), rp, mp, FWD_RTOL, "p'")
    _, rg, rdt = oracle.sgd_bwd(hP, hT if with_dt else None, lr, momentum, nesterov)
    mg, mdt = oracle.sgd_bwd_mag(hP, hT if with_dt else None, lr, momentum, nesterov)
    assert_mag_close(_flat(dg), rg, mg, BWD_RTOL, "dg")
    if mom:
        assert_mag_close(_flat(to), rt, mt, FWD_RTOL, "t'")
        assert_mag_close(_flat(dt), rdt, mdt, BWD_RTOL, "dt")
    # the flat kernels on the flattened tree give the same bits
    f = lambda x: None if x is None else torch.cat([y.reshape(-1) for y in x])  # noqa: E731
    fpo, fto, fdg, fdt = (torch.empty(n, device="cuda") for _ in range(4))
    P.sgd_fwd(f(p), f(g), f(t), lr, momentum, nesterov, fpo, fto if mom else None)
    P.sgd_bwd(f(P_), f(T), lr, momentum, nesterov, fdg, fdt if mom else None)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(po), fpo.view(torch.int32).cpu().numpy())
    assert np.array_equal(_bits(dg), fdg.view(torch.int32).cpu().numpy())
    if mom:
        assert np.array_equal(_bits(to), fto.view(torch.int32).cpu().numpy())
        assert np.array_equal(_bits(dt), fdt.view(torch.int32).cpu().numpy())


@pytest.mark.parametrize("size", ["many", "small"])
@pytest.mark.parametrize("mode", ["separate", "packed-views"])
@pytest.mark.parametrize("momentum,with_b,with_dv,with_db,eps_root", [
    (0.0, False, False, False, 0.0), (0.0, False, True, False, 1e-8), (0.9, False, False, False, 0.0),
    (0.9, True, True, True, 1e-8), (0.9, True, False, True, 0.0), (0.9, True, True, False, 0.0)])
def test_rmsprop_tree_matches_oracle_and_flat(mode, momentum, with_b, with_dv, with_db, eps_root, size):
    import paper_2211_06934_amd as P
    numel = _numel(4, size)
    n = sum(numel)
    table = P.segtable_create(numel)
    lr = 1e-3
    hp, hg = normal(n, 0.05, "rt", "p0", 2), normal(n, 0.01, "rt", "grad", 2)
    hv, hb = abs_normal(n, 1e-4, "rt", "nu", 2), normal(n, 0.1, "rt", "mu", 2)
    hg[:7] = 0.0  # with v = 0 below: the 0/0 point when eps_root = 0
    hv[:3] = 0.0
    hP, hV, hB = (normal(n, 1.0, "rt", s, 2) for s in ("cot_p", "cot_v", "cot_m"))
    tree = lambda a, s: _device_tree(_split(a, numel), mode, s)  # noqa: E731
    p, g, v = tree(hp, 1), tree(hg, 2), tree(hv, 3)
    b = tree(hb, 4) if with_b else None
    P_ = tree(hP, 5)
    V = tree(hV, 6) if with_dv else None
    B = tree(hB, 7) if with_db else None
    mom = momentum > 0
    e = lambda s: _empty_like_tree(p, mode, s)  # noqa: E731
    po, vo, bo = e(8), e(9), (e(10) if mom else None)
    dg, dv, db = e(11), e(12), (e(13) if mom else None)
    pp = lambda x: None if x is None else _ptrs(x)  # noqa: E731
    P.rmsprop_fwd_tree(table, pp(p), pp(g), pp(v), pp(b), lr, ALPHA, EPS, eps_root, momentum, pp(po), pp(vo), pp(bo))
    P.rmsprop_bwd_tree(table, pp(P_), pp(V), pp(B), pp(g), pp(v), lr, ALPHA, EPS, eps_root, momentum, pp(dg), pp(dv),
                       pp(db))
    torch.cuda.synchronize()
    hb_in = hb if with_b else None
    rf = oracle.rmsprop_fwd(hp, hg, hv, hb_in, lr, ALPHA, EPS, eps_root, momentum)
    mf = oracle.rmsprop_fwd_mag(hp, hg, hv, hb_in, lr, ALPHA, EPS, eps_root, momentum)
    assert_mag_close(_flat(po), rf[0], mf[0], FWD_RTOL, "p'")
    assert_mag_close(_flat(vo), rf[1], mf[1], FWD_RTOL, "v'")
    cV, cB = (hV if with_dv else None), (hB if with_db and mom else None)
    rb = oracle.rmsprop_bwd(hP, cV, cB, hg, hv, lr, ALPHA, EPS, eps_root, momentum)
    mb = oracle.rmsprop_bwd_mag(hP, cV, cB, hg, hv, lr, ALPHA, EPS, eps_root, momentum)
    assert_mag_close(_flat(dg), rb[1], mb[0], BWD_RTOL, "dg")
    assert_mag_close(_flat(dv), rb[2], mb[1], BWD_RTOL, "dv")
    if mom:
        assert_mag_close(_flat(bo), rf[2], mf[2], FWD_RTOL, "b'")
        assert_mag_close(_flat(db), rb[3], mb[2], BWD_RTOL, "db")
    f = lambda x: None if x is None else torch.cat([y.reshape(-1) for y in x])  # noqa: E731
    fo = [torch.empty(n, device="cuda") for _ in range(6)]
    P.rmsprop_fwd(f(p), f(g), f(v), f(b), lr, ALPHA, EPS, eps_root, momentum, fo[0], fo[1], fo[2] if mom else None)
    P.rmsprop_bwd(f(P_), f(V), f(B), f(g), f(v), lr, ALPHA, EPS, eps_root, momentum, fo[3], fo[4],
                  fo[5] if mom else None)
    torch.cuda.synchronize()
    pairs = [(po, fo[0]), (vo, fo[1]), (dg, fo[3]), (dv, fo[4])] + ([(bo, fo[2]), (db, fo[5])] if mom else [])
    for tr, fl in pairs:
        assert np.array_equal(_bits(tr), fl.view(torch.int32).cpu().numpy())


def test_optim_tree_invalid_arguments():
    import paper_2211_06934_amd as P
    table = P.segtable_create([4, 5])
    x = [torch.zeros(4, device="cuda"), torch.zeros(5, device="cuda")]
    px = _ptrs(x)
    with pytest.raises(P.DiffoptError, match="momentum"):
        P.sgd_fwd_tree(table, px, px, None, 0.1, -0.5, False, px)
    with pytest.raises(P.DiffoptError, match="null"):
        P.sgd_fwd_tree(table, px, px, None, 0.1, 0.9, False, px, None)  # momentum needs trace_out
    with pytest.raises(P.DiffoptError, match="alpha"):
        P.rmsprop_fwd_tree(table, px, px, px, None, 1e-3, 1.0, EPS, 0.0, 0.0, px, px)
    p1 = _ptrs(x[:1])
    with pytest.raises(P.DiffoptError, match="elem_bytes"):
        P.sgd_fwd_tree(P.segtable_create([4], elem_bytes=8), p1, p1, None, 0.1, 0.0, False, p1)
    torch.cuda.synchronize()


# ------------------------------------------------------------ MAML inner loops


def _meta_grad_ours(which, init, task, K, device, hyper):
    import paper_2211_06934_amd as P
    net = ConvNet(conv_bias=False).to(device)
    with torch.no_grad():
        for nm, prm in net.named_parameters():
            prm.copy_(init[nm])
    p0 = [prm for _, prm in net.named_parameters()]
    opt = P.MetaSGD(net, **hyper) if which == "sgd" else P.MetaRMSProp(net, **hyper)
    xs, ys, xq, yq = (t.to(device) for t in task)
    for _ in range(K):
        opt.step(F.cross_entropy(net(xs), ys))
    outer = F.cross_entropy(net(xq), yq)
    return [g.detach().double().cpu() for g in torch.autograd.grad(outer, p0)], outer.item()


def _meta_grad_reference(which, init, task, K, device, dtype, hyper):
    from torch.optim.rmsprop import rmsprop
    from torch.optim.sgd import sgd
    net = ConvNet(conv_bias=False).to(device=device, dtype=dtype)
    names = [nm for nm, _ in net.named_parameters()]
    p0 = [init[nm].to(device=device, dtype=dtype).clone().requires_grad_() for nm in names]
    params = [prm.clone() for prm in p0]
    zeros = lambda: [torch.zeros_like(prm) for prm in p0]  # noqa: E731
    buf, sq = zeros(), zeros()  # zero-initialised buffers keep the first step differentiable
    xs, ys, xq, yq = (t.to(device=device, dtype=dtype) if t.is_floating_point() else t.to(device) for t in task)

    def fwd(ps, x):
        for nm, prm in zip(names, ps):
            net._parameters[nm] = prm
        return net(x)

    for k in range(K):
        grads = list(torch.autograd.grad(F.cross_entropy(fwd(params, xs), ys), params, create_graph=True))
        params = [prm.clone() for prm in params]
        buf = [x.clone() for x in buf]
        if which == "sgd":
            sgd(params, grads, buf if hyper["momentum"] > 0 else [None] * len(params), weight_decay=0.0,
                momentum=hyper["momentum"], lr=hyper["lr"], dampening=0.0, nesterov=hyper["nesterov"],
                maximize=False)
        else:
            sq = [x.clone() for x in sq]
            rmsprop(params, grads, sq, [], buf if hyper["momentum"] > 0 else [],
                    [torch.tensor(float(k), dtype=dtype) for _ in params], foreach=False, differentiable=True,
                    lr=hyper["lr"], alpha=hyper["alpha"], eps=hyper["eps"], weight_decay=0.0,
                    momentum=hyper["momentum"], centered=False)
    outer = F.cross_entropy(fwd(params, xq), yq)
    return [g.detach().double().cpu() for g in torch.autograd.grad(outer, p0)], outer.item()


@pytest.mark.parametrize("which,hyper", [
    ("sgd", dict(lr=0.1, momentum=0.0, nesterov=False)),
    ("sgd", dict(lr=0.05, momentum=0.9, nesterov=True)),
    ("rmsprop", dict(lr=1e-3, alpha=ALPHA, eps=EPS, momentum=0.0)),
    ("rmsprop", dict(lr=1e-3, alpha=ALPHA, eps=EPS, momentum=0.9)),
])
@pytest.mark.parametrize("K", [1, 3])
def test_maml_meta_gradient_through_fused_sgd_rmsprop(which, hyper, K):
    torch.manual_seed(2)
    init = {nm: prm.detach().clone() for nm, prm in ConvNet(conv_bias=False).named_parameters()}
    task = _task(7)
    ours, out_ours = _meta_grad_ours(which, init, task, K, "cuda", hyper)
    ref64, out64 = _meta_grad_reference(which, init, task, K, "cpu", torch.float64, hyper)
    ref32, _ = _meta_grad_reference(which, init, task, K, "cuda", torch.float32, hyper)
    assert all(torch.isfinite(g).all() for g in ours + ref64 + ref32)
    assert abs(out_ours - out64) <= 1e-4 * abs(out64), (out_ours, out64)
    # Both fp32 loops are nondeterministic through the convolution backward,
    # and the RMSProp meta-gradient is ill-conditioned enough (it divides by
    # sqrt(v)) that single runs of either land anywhere from 2e-2 to 9e-2 from
    # the fp64 loop.  The bar: the nearest of three runs of ours is no further
    # from fp64 than twice the farthest of three runs of torch's loop.  Every
    # step the loop runs is checked element by element against the oracle by
    # test_maml_sgd_rmsprop_steps_match_oracle_inside_the_loop.
    runs = [ours] + [_meta_grad_ours(which, init, task, K, "cuda", hyper)[0] for _ in range(2)]
    e64 = min(_normrel(r, ref64) for r in runs)
    t64 = torch32_spread(lambda: _meta_grad_reference(which, init, task, K, "cuda", torch.float32, hyper)[0], ref64)
    print("%s K=%d  min |ours-fp64|=%.2e  max |torch32-fp64|=%.2e" % (which, K, e64, t64))
    assert e64 < 2 * t64 + 1e-5, (e64, t64)


# ------------------------------------------ every step of the loop vs the oracle

def _cat(ts):
    return np.concatenate([t.detach().reshape(-1).double().cpu().numpy() for t in ts])


def _recording(which, log):
    """SGDTreeFn / RMSPropTreeFn that also record, per call, the fp64 copies of
    what the kernels were given and what they returned."""
    import paper_2211_06934_amd as P
    base = P.autograd.SGDTreeFn if which == "sgd" else P.autograd.RMSPropTreeFn

    class Rec(base):
        @staticmethod
        def forward(ctx, table, hyper, has_state, *leaves):
            out = base.forward(ctx, table, hyper, has_state, *leaves)
            S = len(table.numel)
            torch.cuda.synchronize()
            groups = [_cat(leaves[i * S:(i + 1) * S]) for i in range(len(leaves) // S)]
            log.append(dict(kind="fwd", hyper=hyper, has_state=has_state, inp=groups,
                            out=[_cat(out[i * S:(i + 1) * S]) for i in range(len(out) // S)]))
            return out

        @staticmethod
        def backward(ctx, *cots):
            res = base.backward(ctx, *cots)
            S = ctx.S
            torch.cuda.synchronize()
            like = res[3:3 + S]  # dP: shapes of the params
            grp = lambda k: None if all(c is None for c in cots[k * S:(k + 1) * S]) else \
                _cat([torch.zeros_like(x) if c is None else c for c, x in zip(cots[k * S:(k + 1) * S], like)])  # noqa
            rec = dict(kind="bwd", hyper=ctx.hyper, cots=[grp(k) for k in range(len(cots) // S)],
                       res=[None if r[0] is None else _cat(r) for r in
                            (res[3 + k * S:3 + (k + 1) * S] for k in range((len(res) - 3) // S))])
            if which == "rmsprop":
                saved = ctx.saved_tensors
                rec["g"], rec["v"] = _cat(saved[:S]), _cat(saved[S:])
            log.append(rec)
            return res

    return Rec


@pytest.mark.parametrize("which,hyper", [
    ("sgd", dict(lr=0.05, momentum=0.9, nesterov=True)),
    ("sgd", dict(lr=0.1, momentum=0.0, nesterov=False)),
    ("rmsprop", dict(lr=1e-3, alpha=ALPHA, eps=EPS, momentum=0.0)),
    ("rmsprop", dict(lr=1e-3, alpha=ALPHA, eps=EPS, momentum=0.9)),
])
@pytest.mark.parametrize("K", [1, 3])
def test_maml_sgd_rmsprop_steps_match_oracle_inside_the_loop(which, hyper, K, monkeypatch):
    # every fused step MetaSGD / MetaRMSProp runs inside the MAML loop --
    # warm states after step 1, cotangents carrying the model's second-order
    # terms -- element by element against the oracle on the inputs that step
    # received: 1e-5 of the term scale forward, 1e-4 for the VJP, and the
    # params cotangent passed through bit for bit
    import oracle
    import paper_2211_06934_amd as P
    log = []
    name = "SGDTreeFn" if which == "sgd" else "RMSPropTreeFn"
    monkeypatch.setattr(P.autograd, name, _recording(which, log))
    torch.manual_seed(2 + K)
    init = {nm: prm.detach().clone() for nm, prm in ConvNet(conv_bias=False).named_parameters()}
    grads, outer = _meta_grad_ours(which, init, _task(7 + K), K, "cuda", hyper)
    assert np.isfinite(outer) and all(torch.isfinite(g).all() for g in grads)
    fw = [r for r in log if r["kind"] == "fwd"]
    bw = [r for r in log if r["kind"] == "bwd"]
    assert len(fw) == K and len(bw) == K
    mom = hyper["momentum"] > 0
    for k, r in enumerate(fw):
        h = r["hyper"]
        if which == "sgd":
            p, g = r["inp"][:2]
            t = r["inp"][2] if r["has_state"] else None
            args = (h.lr, h.momentum, h.nesterov)
            ref, mag = oracle.sgd_fwd(p, g, t, *args), oracle.sgd_fwd_mag(p, g, t, *args)
            names = ("p'", "t'")
        else:
            p, g, v = r["inp"][:3]
            b = r["inp"][3] if r["has_state"] else None
            args = (h.lr, h.alpha, h.eps, h.eps_root, h.momentum)
            ref, mag = oracle.rmsprop_fwd(p, g, v, b, *args), oracle.rmsprop_fwd_mag(p, g, v, b, *args)
            names = ("p'", "v'", "b'")
        for nm, got, x, mg in zip(names, r["out"], ref, mag):
            assert_mag_close(got, x, mg, FWD_RTOL, "%s step %d %s" % (which, k, nm))
    for r in bw:
        h = r["hyper"]
        if which == "sgd":
            dP = r["cots"][0] if r["cots"][0] is not None else np.zeros_like(r["res"][0])
            dT = r["cots"][1] if mom and len(r["cots"]) > 1 else None
            args = (h.lr, h.momentum, h.nesterov)
            _, rg, rdt = oracle.sgd_bwd(dP, dT, *args)
            mg, mdt = oracle.sgd_bwd_mag(dP, dT, *args)
            checks = [("dg", r["res"][1], rg, mg)]
            if mom and len(r["res"]) > 2 and r["res"][2] is not None:  # a trace was an input of this step
                checks.append(("dt", r["res"][2], rdt, mdt))
        else:
            dP = r["cots"][0] if r["cots"][0] is not None else np.zeros_like(r["g"])
            dV = r["cots"][1]
            dB = r["cots"][2] if mom else None
            args = (h.lr, h.alpha, h.eps, h.eps_root, h.momentum)
            _, rg, rdv, rdb = oracle.rmsprop_bwd(dP, dV, dB, r["g"], r["v"], *args)
            mg, mdv, mdb = oracle.rmsprop_bwd_mag(dP, dV, dB, r["g"], r["v"], *args)
            checks = [("dg", r["res"][1], rg, mg), ("dv", r["res"][2], rdv, mdv)]
            if mom and len(r["res"]) > 3 and r["res"][3] is not None:
                checks.append(("db", r["res"][3], rdb, mdb))
        assert np.array_equal(r["res"][0], dP), "params cotangent is the identity"
        for nm, got, x, mg in checks:
            assert_mag_close(got, x, mg, BWD_RTOL, "%s VJP %s" % (which, nm))
