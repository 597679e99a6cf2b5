"""GPU parity of the leaf-direct ("tree map") Adam step and its K-step driver.

By definition the tree-map step equals flatten -> flat step -> unflatten, so
the expected values are the oracle's flat step applied to the oracle's pack of
the leaves, split back with the oracle's unpack.  Trees cover empty and tiny
leaves, ragged sizes, leaves out of 16-byte phase (element path), in-place
aliasing, and the 20,000-leaf workload at full size (sampled leaves).
"""
import numpy as np
import pytest
import torch

import oracle
from tests.support import BWD_RTOL, FWD_RTOL, assert_mag_close, stats
from workloads import HYPER, many_small, normal, abs_normal, random_shapes

pytestmark = pytest.mark.gpu

LR, B1, B2, EPS = HYPER["lr"], HYPER["b1"], HYPER["b2"], HYPER["eps"]


def _ptrs(leaves):
    return torch.tensor([x.data_ptr() for x in leaves], dtype=torch.int64, device="cuda")


def _device_tree(host_leaves, mode, seed):
    """Device copies: separate allocations, or views at random element offsets
    inside one buffer (leaves out of 16-byte phase)."""
    numel = [x.size for x in host_leaves]
    flat = torch.from_numpy(np.concatenate([x.reshape(-1) for x in host_leaves]).astype(np.float32)).cuda() \
        if host_leaves else torch.zeros(0, device="cuda")
    if mode == "separate":
        return [x.clone() for x in torch.split(flat, numel)]
    rng = np.random.default_rng(seed)
    total = sum(numel) + 8 * (len(numel) + 1)
    big = torch.zeros(total, dtype=torch.float32, device="cuda")
    out, pos, src = [], int(rng.integers(0, 4)), 0
    for k in numel:
        v = big[pos:pos + k]
        v.copy_(flat[src:src + k])
        out.append(v)
        src += k
        pos += k + int(rng.integers(0, 5))
    return out


def _empty_like_tree(tree, mode, seed):
    if mode == "separate":
        return [torch.empty(x.numel(), device="cuda") for x in tree]
    rng = np.random.default_rng(seed)
    total = sum(x.numel() for x in tree) + 8 * (len(tree) + 1)
    big = torch.zeros(total, dtype=torch.float32, device="cuda")
    out, pos = [], int(rng.integers(0, 4))
    for x in tree:
        out.append(big[pos:pos + x.numel()])
        pos += x.numel() + int(rng.integers(0, 5))
    return out


def _host(tree):
    return [x.cpu().numpy() for x in tree]


def _split(flat, numel):
    return np.split(np.asarray(flat), np.cumsum(numel)[:-1]) if numel else []


def _leaves(numel, seed, moments):
    n = int(sum(numel))
    p = normal(n, 0.05, "tm", "p0", seed)
    g = normal(n, 0.01, "tm", "grad", seed)
    m = normal(n, 1e-3, "tm", "mu", seed) if moments else np.zeros(n, np.float32)
    v = abs_normal(n, 1e-4, "tm", "nu", seed) if moments else np.zeros(n, np.float32)
    cots = [normal(n, 1.0, "tm", t, seed) for t in ("cot_p", "cot_m", "cot_v")]
    return [_split(a, numel) for a in (p, g, m, v, *cots)]


@pytest.mark.parametrize("mode", ["separate", "packed-views"])
@pytest.mark.parametrize("count,moments,eps_root", [(0, False, 0.0), (7, True, 1e-8)])
def test_tree_fwd_bwd_match_oracle(mode, count, moments, eps_root):
    import paper_2211_06934_amd as P
    shapes = random_shapes(300, 4000, seed=17)
    numel = [int(np.prod(s)) for s in shapes]
    table = P.segtable_create(numel)
    hp, hg, hm, hv, hP, hM, hV = _leaves(numel, 3, moments)
    T = {name: _device_tree(h, mode, i) for i, (name, h) in
         enumerate((("p", hp), ("g", hg), ("m", hm), ("v", hv), ("P", hP), ("M", hM), ("V", hV)))}
    out = {name: _empty_like_tree(T["p"], mode, 10 + i) for i, name in enumerate(("po", "mo", "vo", "dg", "dm", "dv"))}
    ptr = {k: _ptrs(v) for k, v in {**T, **out}.items()}
    P.adam_fwd_tree(table, ptr["p"], ptr["g"], ptr["m"], ptr["v"], count, LR, B1, B2, EPS, eps_root,
                    ptr["po"], ptr["mo"], ptr["vo"])
    P.adam_bwd_tree(table, ptr["P"], ptr["M"], ptr["V"], ptr["g"], ptr["m"], ptr["v"], count, LR, B1, B2, EPS,
                    eps_root, ptr["dg"], ptr["dm"], ptr["dv"])
    torch.cuda.synchronize()
    flat = {k: oracle.pack(h).astype(np.float64) for k, h in
            (("p", hp), ("g", hg), ("m", hm), ("v", hv), ("P", hP), ("M", hM), ("V", hV))}
    ref = oracle.adam_fwd(flat["p"], flat["g"], flat["m"], flat["v"], count, LR, B1, B2, EPS, eps_root)
    mag = oracle.adam_fwd_mag(flat["p"], flat["g"], flat["m"], flat["v"], count, LR, B1, B2, EPS, eps_root)
    for name, r, mg in zip(("po", "mo", "vo"), ref, mag):
        got = np.concatenate(_host(out[name])) if numel else np.zeros(0)
        assert_mag_close(got, r, mg, FWD_RTOL, name)
    refb = oracle.adam_bwd(flat["P"], flat["M"], flat["V"], flat["g"], flat["m"], flat["v"], count, LR, B1, B2,
                           EPS, eps_root)
    magb = oracle.adam_bwd_mag(flat["P"], flat["M"], flat["V"], flat["g"], flat["m"], flat["v"], count, LR, B1,
                               B2, EPS, eps_root)
    for name, r, mg in zip(("dg", "dm", "dv"), refb[1:], magb):
        got = np.concatenate(_host(out[name]))
        assert_mag_close(got, r, mg, BWD_RTOL, name)
    table.close()


def test_tree_bwd_without_moment_cotangents_and_in_place():
    import paper_2211_06934_amd as P
    numel = [int(np.prod(s)) for s in random_shapes(200, 3000, seed=23)]
    table = P.segtable_create(numel)
    hp, hg, hm, hv, hP, _, _ = _leaves(numel, 4, True)
    p, g, m, v, dP = (_device_tree(h, "separate", 0) for h in (hp, hg, hm, hv, hP))
    # forward in place over p, m, v
    P.adam_fwd_tree(table, _ptrs(p), _ptrs(g), _ptrs(m), _ptrs(v), 3, LR, B1, B2, EPS, 0.0,
                    _ptrs(p), _ptrs(m), _ptrs(v))
    dg, dm, dv = (_empty_like_tree(p, "separate", 0) for _ in range(3))
    g0, m0, v0 = (_device_tree(h, "separate", 0) for h in (hg, hm, hv))
    P.adam_bwd_tree(table, _ptrs(dP), None, None, _ptrs(g0), _ptrs(m0), _ptrs(v0), 3, LR, B1, B2, EPS, 0.0,
                    _ptrs(dg), _ptrs(dm), _ptrs(dv))
    torch.cuda.synchronize()
    F = [oracle.pack(h).astype(np.float64) for h in (hp, hg, hm, hv, hP)]
    ref = oracle.adam_fwd(F[0], F[1], F[2], F[3], 3, LR, B1, B2, EPS, 0.0)
    mag = oracle.adam_fwd_mag(F[0], F[1], F[2], F[3], 3, LR, B1, B2, EPS, 0.0)
    for name, t, r, mg in zip(("p", "m", "v"), (p, m, v), ref, mag):
        assert_mag_close(np.concatenate(_host(t)), r, mg, FWD_RTOL, name)
    refb = oracle.adam_bwd(F[4], None, None, F[1], F[2], F[3], 3, LR, B1, B2, EPS, 0.0)
    magb = oracle.adam_bwd_mag(F[4], None, None, F[1], F[2], F[3], 3, LR, B1, B2, EPS, 0.0)
    for name, t, r, mg in zip(("dg", "dm", "dv"), (dg, dm, dv), refb[1:], magb):
        assert_mag_close(np.concatenate(_host(t)), r, mg, BWD_RTOL, name)


def _unrolled_tree(P, table, numel, K, seed, mode, count0=0, eps_root=0.0):
    n = int(sum(numel))
    G = np.stack([normal(n, 0.01, "tmu", "grad", 100 * seed + k) for k in range(K)])
    p0 = normal(n, 0.05, "tmu", "p0", seed)
    cot = normal(n, 1.0, "tmu", "cot_p", seed)
    z = np.zeros(n, np.float32)
    trees = dict(p0=_device_tree(_split(p0, numel), mode, 1), cot=_device_tree(_split(cot, numel), mode, 2),
                 g=[_device_tree(_split(G[k], numel), mode, 3 + k) for k in range(K)],
                 mu=[_device_tree(_split(z, numel), mode, 20)],
                 nu=[_device_tree(_split(z, numel), mode, 40)])
    trees["mu"] += [_empty_like_tree(trees["mu"][0], mode, 21 + k) for k in range(K)]
    trees["nu"] += [_empty_like_tree(trees["nu"][0], mode, 41 + k) for k in range(K)]
    trees["pK"] = _empty_like_tree(trees["p0"], mode, 60)
    trees["dg"] = [_empty_like_tree(trees["p0"], mode, 61 + k) for k in range(K)]
    trees["dm0"] = _empty_like_tree(trees["p0"], mode, 80)
    trees["dv0"] = _empty_like_tree(trees["p0"], mode, 81)
    pt = lambda t: _ptrs(t)  # noqa: E731
    args = (count0, LR, B1, B2, EPS, eps_root)
    P.adam_unrolled_fwd_tree(table, pt(trees["p0"]), [pt(t) for t in trees["g"]], [pt(t) for t in trees["mu"]],
                             [pt(t) for t in trees["nu"]], pt(trees["pK"]), *args)
    P.adam_unrolled_bwd_tree(table, pt(trees["cot"]), [pt(t) for t in trees["g"]], [pt(t) for t in trees["mu"]],
                             [pt(t) for t in trees["nu"]], [pt(t) for t in trees["dg"]], pt(trees["dm0"]),
                             pt(trees["dv0"]), *args)
    torch.cuda.synchronize()
    return trees, p0, G, cot


@pytest.mark.parametrize("mode", ["separate", "packed-views"])
def test_unrolled_tree_matches_oracle(mode):
    import paper_2211_06934_amd as P
    numel = [int(np.prod(s)) for s in random_shapes(150, 5000, seed=29)]
    K = 4
    table = P.segtable_create(numel)
    trees, p0, G, cot = _unrolled_tree(P, table, numel, K, 5, mode)
    n = int(sum(numel))
    z = np.zeros(n)
    # local forward on the GPU's own trajectory, then p_K and the meta-gradient
    mt = np.stack([np.concatenate(_host(t)) for t in trees["mu"]]).astype(np.float64)
    vt = np.stack([np.concatenate(_host(t)) for t in trees["nu"]]).astype(np.float64)
    for k in range(1, K + 1):
        r = oracle.adam_fwd(p0, G[k - 1], mt[k - 1], vt[k - 1], k - 1, LR, B1, B2, EPS, 0.0)
        mg = oracle.adam_fwd_mag(p0, G[k - 1], mt[k - 1], vt[k - 1], k - 1, LR, B1, B2, EPS, 0.0)
        assert_mag_close(mt[k], r[1], mg[1], FWD_RTOL, "m_%d" % k)
        assert_mag_close(vt[k], r[2], mg[2], FWD_RTOL, "v_%d" % k)
    pK_ref, mt_ref, vt_ref = oracle.unrolled_fwd(p0, G, z, z, 0, LR, B1, B2, EPS, 0.0)
    assert stats(np.concatenate(_host(trees["pK"])), pK_ref)[1] < FWD_RTOL
    _, dg_l, dm_l, dv_l = oracle.unrolled_bwd(cot, G, mt, vt, 0, LR, B1, B2, EPS, 0.0)
    magM = np.zeros(n)
    magV = np.zeros(n)
    for k in range(K, 0, -1):
        mg, mm, mv = oracle.adam_bwd_mag(cot, magM, magV, G[k - 1], mt[k - 1], vt[k - 1], k - 1, LR, B1, B2, EPS,
                                         0.0)
        assert_mag_close(np.concatenate(_host(trees["dg"][k - 1])), dg_l[k - 1], mg, BWD_RTOL, "dg_%d" % k)
        magM, magV = mm, mv
    assert_mag_close(np.concatenate(_host(trees["dm0"])), dm_l, magM, BWD_RTOL, "dm0")
    assert_mag_close(np.concatenate(_host(trees["dv0"])), dv_l, magV, BWD_RTOL, "dv0")


def test_tree_map_equals_flat_path_on_gpu():
    # property: the leaf-direct step and flatten -> flat step agree element for
    # element (same arithmetic per element); checked against each other and
    # both against the oracle's bound
    import paper_2211_06934_amd as P
    numel = [int(np.prod(s)) for s in random_shapes(120, 6000, seed=31)]
    table = P.segtable_create(numel)
    hp, hg, hm, hv, _, _, _ = _leaves(numel, 8, True)
    p, g, m, v = (_device_tree(h, "separate", 0) for h in (hp, hg, hm, hv))
    po, mo, vo = (_empty_like_tree(p, "separate", 0) for _ in range(3))
    P.adam_fwd_tree(table, _ptrs(p), _ptrs(g), _ptrs(m), _ptrs(v), 11, LR, B1, B2, EPS, 1e-8,
                    _ptrs(po), _ptrs(mo), _ptrs(vo))
    n = int(sum(numel))
    flat_in = [torch.empty(n, device="cuda") for _ in range(4)]
    for f, t in zip(flat_in, (p, g, m, v)):
        P.tree_flatten(table, _ptrs(t), f)
    flat_out = [torch.empty(n, device="cuda") for _ in range(3)]
    P.adam_fwd(*flat_in, 11, LR, B1, B2, EPS, 1e-8, *flat_out)
    torch.cuda.synchronize()
    for t, f in zip((po, mo, vo), flat_out):
        got = torch.cat([x.reshape(-1) for x in t]).cpu().numpy().astype(np.float64)
        ref = f.cpu().numpy().astype(np.float64)
        assert np.max(np.abs(got - ref) / np.maximum(np.abs(ref), 1e-30)) < 1e-6


def test_unrolled_tree_many_small_full_size_sampled_leaves():
    import paper_2211_06934_amd as P
    w = many_small()
    numel = w.numels
    K = w.K
    table = P.segtable_create(numel)
    trees, p0, G, cot = _unrolled_tree(P, table, numel, K, 7, "separate")
    rng = np.random.default_rng(11)
    pick = sorted(set([0, 1, len(numel) - 1] + list(rng.integers(0, len(numel), size=300))))
    offs = np.concatenate([[0], np.cumsum(numel)])
    idx = np.concatenate([np.arange(offs[j], offs[j + 1]) for j in pick])
    z = np.zeros(idx.size)
    Gs = G[:, idx].astype(np.float64)
    pK_ref, mt_ref, vt_ref = oracle.unrolled_fwd(p0[idx], Gs, z, z, 0, LR, B1, B2, EPS, 0.0)
    _, dg_ref, dm_ref, dv_ref = oracle.unrolled_bwd(cot[idx], Gs, mt_ref, vt_ref, 0, LR, B1, B2, EPS, 0.0)

    def gather(tree):
        return np.concatenate([tree[j].cpu().numpy() for j in pick]).astype(np.float64)

    assert stats(gather(trees["pK"]), pK_ref)[1] < FWD_RTOL
    for k in range(K):
        assert stats(gather(trees["dg"][k]), dg_ref[k])[1] < BWD_RTOL
    assert stats(gather(trees["dm0"]), dm_ref)[1] < BWD_RTOL
    assert stats(gather(trees["dv0"]), dv_ref)[1] < BWD_RTOL
