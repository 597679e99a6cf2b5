"""GPU parity of the leaf-direct Adam kernels on small trees (at most 32
nonempty leaves and 2^16 elements), which take one element per lane with the
leaf table in kernel arguments.

Each case runs the same leaves through a small table and through a table that
also holds 33 more leaves (so it takes the tiled kernels), and requires every
output on the shared leaves to agree bit for bit: the per-element arithmetic
is the same in both forms.  The tiled form is compared with the oracle by
tests/test_gpu_treemap.py and tests/test_gpu_treemap_fused.py; here the small
form is also compared with the oracle directly.  Trees hold empty leaves,
ragged sizes and leaves out of 16-byte phase; the table sizes straddle both
limits (32 / 33 leaves, 2^16 / 2^16 + 1 elements).
"""
import numpy as np
import pytest
import torch

import oracle
from tests.support import BWD_RTOL, FWD_RTOL, assert_mag_close
from tests.test_gpu_treemap import _device_tree, _empty_like_tree, _leaves, _ptrs
from workloads import HYPER

pytestmark = pytest.mark.gpu

LR, B1, B2, EPS = HYPER["lr"], HYPER["b1"], HYPER["b2"], HYPER["eps"]
PAD = [5, 0, 17, 64, 1, 3, 100, 2, 9, 31, 8, 4, 77, 6, 13, 0, 40, 2, 11, 1, 19, 7, 25, 3, 16, 5, 2, 61, 9, 1, 33,
       4, 12, 7]  # 33 nonempty leaves: any table holding them takes the tiled kernels

SMALL = {
    "ragged": [0, 3, 40, 1, 1600, 0, 40, 7, 1, 4096, 5, 2, 0],
    "32-leaves": [(7 * k) % 23 + 1 for k in range(32)],
    "2^16-elements": [1 << 15, 1, (1 << 15) - 4, 3],
    # 40 leaves of which 26 are empty: the small form, with caller leaf
    # indices up to 39 (past the table's 32 slots)
    "sparse": [0 if k % 4 else 3 * k + 1 for k in range(40)][:30] + [5, 0, 9, 0, 2, 0, 7, 0, 11, 4],
}


def _inputs(numel, K, mode, seed):
    hp, _, hm, hv, hc, _, _ = _leaves(numel, seed, True)
    T = dict(p0=_device_tree(hp, mode, seed), m0=_device_tree(hm, mode, seed + 1),
             v0=_device_tree(hv, mode, seed + 2), cot=_device_tree(hc, mode, seed + 3))
    T["G"] = [_device_tree(_leaves(numel, seed * 100 + k, False)[1], mode, seed + 10 + k) for k in range(K)]
    return T


def _run(P, table, S, T, K, count0, er, in_place, fused, keep):
    """The K-step pass over the first S leaves of the trees in T (fresh output
    trees; p0 cloned when it is updated in place).  keep: the intermediate
    states stored (None: all of them)."""
    cut = lambda t: t[:S]  # noqa: E731
    new = lambda: [torch.full_like(x, float("nan")) for x in cut(T["p0"])]  # noqa: E731
    stored = lambda k: keep is None or k in keep or k == K  # noqa: E731
    p0 = [x.clone() for x in cut(T["p0"])]
    mu = [cut(T["m0"])] + [new() if stored(k + 1) else None for k in range(K)]
    nu = [cut(T["v0"])] + [new() if stored(k + 1) else None for k in range(K)]
    pK = p0 if in_place else new()
    dg = [new() for _ in range(K)]
    dm0, dv0 = new(), new()
    G = [cut(g) for g in T["G"]]
    cot = cut(T["cot"])
    if fused:
        mp = [None if t is None else _ptrs(t) for t in mu]
        vp = [None if t is None else _ptrs(t) for t in nu]
        P.adam_unrolled_fwd_tree(table, _ptrs(p0), [_ptrs(g) for g in G], mp, vp, _ptrs(pK), count0, LR, B1, B2,
                                 EPS, er)
        P.adam_unrolled_bwd_tree(table, _ptrs(cot), [_ptrs(g) for g in G], mp, vp, [_ptrs(t) for t in dg],
                                 _ptrs(dm0), _ptrs(dv0), count0, LR, B1, B2, EPS, er)
    else:
        src = p0
        for k in range(K):
            P.adam_fwd_tree(table, _ptrs(src), _ptrs(G[k]), _ptrs(mu[k]), _ptrs(nu[k]), count0 + k, LR, B1, B2,
                            EPS, er, _ptrs(pK), _ptrs(mu[k + 1]), _ptrs(nu[k + 1]))
            src = pK
        for k in range(K - 1, -1, -1):
            first = k == K - 1
            P.adam_bwd_tree(table, _ptrs(cot), None if first else _ptrs(dm0), None if first else _ptrs(dv0),
                            _ptrs(G[k]), _ptrs(mu[k]), _ptrs(nu[k]), count0 + k, LR, B1, B2, EPS, er,
                            _ptrs(dg[k]), _ptrs(dm0), _ptrs(dv0))
    torch.cuda.synchronize()
    return dict(pK=pK, mu=mu[1:], nu=nu[1:], dg=dg, dm0=dm0, dv0=dv0)


def _bits(tree):
    if not tree:
        return np.zeros(0, np.int32)
    return torch.cat([x.reshape(-1) for x in tree]).view(torch.int32).cpu().numpy()


def _same(a, b, what):
    x, y = _bits(a), _bits(b)
    assert x.size == y.size, what
    bad = np.flatnonzero(x != y)
    assert bad.size == 0, "%s: %d of %d differ, first at %d" % (what, bad.size, x.size, bad[0])


def _compare(small, big, K):
    _same(small["pK"], big["pK"], "p_K")
    for k in range(K):
        if small["mu"][k] is not None:
            _same(small["mu"][k], big["mu"][k], "mu_%d" % (k + 1))
            _same(small["nu"][k], big["nu"][k], "nu_%d" % (k + 1))
        _same(small["dg"][k], big["dg"][k], "dg_%d" % (k + 1))
    _same(small["dm0"], big["dm0"], "dmu0")
    _same(small["dv0"], big["dv0"], "dnu0")


@pytest.mark.parametrize("tree", list(SMALL))
@pytest.mark.parametrize("K,count0,er,mode,in_place,fused,keep", [
    (1, 0, 0.0, "separate", False, True, None),
    (1, 7, 1e-8, "packed-views", True, False, None),      # single steps, in place, out of phase
    (3, 5, 1e-8, "packed-views", False, False, None),
    (5, 0, 0.0, "separate", False, True, ()),             # one recomputed run (the benchmark's form)
    (5, 2, 1e-8, "packed-views", True, True, None),       # stored trajectory: tiled VJP kernel, small forward
    (8, 0, 1e-8, "separate", True, True, ()),             # the longest run in one launch
    (10, 1, 0.0, "packed-views", False, True, (8,)),      # two launches each way, runs of 8 and 2 recomputed
    (11, 0, 1e-8, "separate", False, True, (3, 10)),      # recomputed and stored runs mixed
])
def test_small_tree_equals_tiled_kernels_bitwise(tree, K, count0, er, mode, in_place, fused, keep):
    import paper_2211_06934_amd as P
    numel = SMALL[tree]
    S = len(numel)
    T = _inputs(numel + PAD, K, mode, 3 + K)
    small_table = P.segtable_create(numel)
    big_table = P.segtable_create(numel + PAD)
    keep = None if keep is None else set(keep)
    got = _run(P, small_table, S, T, K, count0, er, in_place, fused, keep)
    ref = _run(P, big_table, len(numel) + len(PAD), T, K, count0, er, in_place, fused, keep)
    for name in ("pK", "dm0", "dv0"):
        ref[name] = ref[name][:S]
    for name in ("mu", "nu", "dg"):
        ref[name] = [None if t is None else t[:S] for t in ref[name]]
    _compare(got, ref, K)
    small_table.close()
    big_table.close()


@pytest.mark.parametrize("numel", [SMALL["ragged"], [1 << 16], [(1 << 16) + 1], SMALL["32-leaves"] + [2]])
def test_table_limits_single_step_matches_oracle(numel):
    # the single step and its VJP, with and without incoming moment
    # cotangents, against the oracle's flat step on the packed leaves; the
    # sizes sit on both sides of each limit of the small form
    import paper_2211_06934_amd as P
    count, er = 4, 1e-8
    table = P.segtable_create(numel)
    hp, hg, hm, hv, hP, hM, hV = _leaves(numel, 21, True)
    dev = {k: _device_tree(h, "separate", i) for i, (k, h) in
           enumerate((("p", hp), ("g", hg), ("m", hm), ("v", hv), ("P", hP), ("M", hM), ("V", hV)))}
    out = {k: _empty_like_tree(dev["p"], "separate", 0) for k in ("po", "mo", "vo", "dg", "dm", "dv", "dg0", "dm0",
                                                                  "dv0")}
    ptr = {k: _ptrs(v) for k, v in {**dev, **out}.items()}
    P.adam_fwd_tree(table, ptr["p"], ptr["g"], ptr["m"], ptr["v"], count, LR, B1, B2, EPS, er,
                    ptr["po"], ptr["mo"], ptr["vo"])
    P.adam_bwd_tree(table, ptr["P"], ptr["M"], ptr["V"], ptr["g"], ptr["m"], ptr["v"], count, LR, B1, B2, EPS, er,
                    ptr["dg"], ptr["dm"], ptr["dv"])
    P.adam_bwd_tree(table, ptr["P"], None, None, ptr["g"], ptr["m"], ptr["v"], count, LR, B1, B2, EPS, er,
                    ptr["dg0"], ptr["dm0"], ptr["dv0"])
    torch.cuda.synchronize()
    got = {k: torch.cat([x.reshape(-1) for x in t]).cpu().numpy().astype(np.float64) for k, t in out.items()}
    flat = {k: oracle.pack(h).astype(np.float64) for k, h in
            (("p", hp), ("g", hg), ("m", hm), ("v", hv), ("P", hP), ("M", hM), ("V", hV))}
    z = np.zeros_like(flat["p"])
    ref = oracle.adam_fwd(flat["p"], flat["g"], flat["m"], flat["v"], count, LR, B1, B2, EPS, er)
    mag = oracle.adam_fwd_mag(flat["p"], flat["g"], flat["m"], flat["v"], count, LR, B1, B2, EPS, er)
    for name, r, mg in zip(("po", "mo", "vo"), ref, mag):
        assert_mag_close(got[name], r, mg, FWD_RTOL, name)
    for suffix, (M, V) in (("", (flat["M"], flat["V"])), ("0", (z, z))):
        refb = oracle.adam_bwd(flat["P"], M, V, flat["g"], flat["m"], flat["v"], count, LR, B1, B2, EPS, er)
        magb = oracle.adam_bwd_mag(flat["P"], M, V, flat["g"], flat["m"], flat["v"], count, LR, B1, B2, EPS, er)
        for name, r, mg in zip(("dg", "dm", "dv"), refb[1:], magb):
            assert_mag_close(got[name + suffix], r, mg, BWD_RTOL, name + suffix)
    table.close()


def test_small_tree_fused_matches_oracle():
    # K = 5 from zero moments with nothing stored between the initial and
    # final states (the benchmark's tiny-MLP form): p_K, the final moments
    # and every meta-gradient against the oracle's unrolled pass
    import paper_2211_06934_amd as P
    numel = [40, 40, 1600, 40, 40, 1]
    K = 5
    table = P.segtable_create(numel)
    hp, _, _, _, hc, _, _ = _leaves(numel, 31, False)
    p0 = _device_tree(hp, "separate", 0)
    cot = _device_tree(hc, "separate", 1)
    Gh = [_leaves(numel, 500 + k, False)[1] for k in range(K)]
    G = [_device_tree(g, "separate", 2 + k) for k, g in enumerate(Gh)]
    zero = lambda: [torch.zeros_like(x) for x in p0]  # noqa: E731
    new = lambda: [torch.empty_like(x) for x in p0]  # noqa: E731
    mu = [zero()] + [None] * (K - 1) + [new()]
    nu = [zero()] + [None] * (K - 1) + [new()]
    pK, dg, dm0, dv0 = new(), [new() for _ in range(K)], new(), new()
    mp = [None if t is None else _ptrs(t) for t in mu]
    vp = [None if t is None else _ptrs(t) for t in nu]
    P.adam_unrolled_fwd_tree(table, _ptrs(p0), [_ptrs(g) for g in G], mp, vp, _ptrs(pK), 0, LR, B1, B2, EPS, 0.0)
    P.adam_unrolled_bwd_tree(table, _ptrs(cot), [_ptrs(g) for g in G], mp, vp, [_ptrs(t) for t in dg],
                             _ptrs(dm0), _ptrs(dv0), 0, LR, B1, B2, EPS, 0.0)
    torch.cuda.synchronize()
    cat = lambda t: torch.cat([x.reshape(-1) for x in t]).cpu().numpy().astype(np.float64)  # noqa: E731
    fp0, fcot = oracle.pack(hp).astype(np.float64), oracle.pack(hc).astype(np.float64)
    fG = np.stack([oracle.pack(g).astype(np.float64) for g in Gh])
    n = fp0.size
    z = np.zeros(n)
    pK_ref, mt, vt = oracle.unrolled_fwd(fp0, fG, z, z, 0, LR, B1, B2, EPS, 0.0)
    # p_K = p_0 minus K updates: its scale is |p_0| plus the K update scales;
    # each moment recurrence's scale is summed the same way
    mag_p, mag_m, mag_v = np.abs(fp0), z, z
    for k in range(K):
        mg = oracle.adam_fwd_mag(fp0, fG[k], mt[k], vt[k], k, LR, B1, B2, EPS, 0.0)
        mag_p = mag_p + mg[3]
        mag_m = B1 * mag_m + (1 - B1) * np.abs(fG[k])
        mag_v = B2 * mag_v + (1 - B2) * fG[k] ** 2
    assert_mag_close(cat(pK), pK_ref, mag_p, FWD_RTOL, "p_K")
    assert_mag_close(cat(mu[K]), mt[K], mag_m, FWD_RTOL, "mu_K")
    assert_mag_close(cat(nu[K]), vt[K], mag_v, FWD_RTOL, "nu_K")
    _, dg_l, dm_l, dv_l = oracle.unrolled_bwd(fcot, fG, mt, vt, 0, LR, B1, B2, EPS, 0.0)
    magM, magV = z, z
    for k in range(K, 0, -1):
        mg, mm, mv = oracle.adam_bwd_mag(fcot, magM, magV, fG[k - 1], mt[k - 1], vt[k - 1], k - 1, LR, B1, B2, EPS,
                                         0.0)
        assert_mag_close(cat(dg[k - 1]), dg_l[k - 1], mg, BWD_RTOL, "dg_%d" % k)
        magM, magV = mm, mv
    assert_mag_close(cat(dm0), dm_l, magM, BWD_RTOL, "dm0")
    assert_mag_close(cat(dv0), dv_l, magV, BWD_RTOL, "dv0")
    table.close()
