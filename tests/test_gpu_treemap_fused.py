"""The leaf-direct K-step driver runs its steps fused, up to 8 per launch, with
each lane's running state in registers.  Each step's arithmetic is that of the
single-step leaf-direct kernels, in the same order, so the fused driver must
reproduce the step-by-step composition of diffopt_adam_fwd_tree /
diffopt_adam_bwd_tree bit for bit: across launch chunks (K = 8, 9, 17), with
empty leaves, leaves out of 16-byte phase (element path), nonzero initial
moments and in-place p_K == p0.

With intermediate trajectory entries left NULL, the VJP recomputes those
states from the latest stored one; the results must equal the fully stored
run bit for bit, across the forward's 8-step launch boundaries (where the
running moments pass through the final-state trees) and at the 20,000-leaf
benchmark size."""
import numpy as np
import pytest
import torch

from tests.test_gpu_treemap import _device_tree, _empty_like_tree, _leaves, _ptrs
from workloads import HYPER, random_shapes

pytestmark = pytest.mark.gpu

LR, B1, B2, EPS = HYPER["lr"], HYPER["b1"], HYPER["b2"], HYPER["eps"]


def _numel(seed):
    shapes = random_shapes(90, 3000, seed=seed)
    numel = [int(np.prod(s)) for s in shapes]
    return [0, 3] + numel[:40] + [0, 0, 1, 4096, 5] + numel[40:]


def _grads(numel, K, mode, seed):
    out = []
    for k in range(K):
        _, hg, _, _, _, _, _ = _leaves(numel, seed * 100 + k, False)
        out.append(_device_tree(hg, mode, seed + k))
    return out


def _run(P, table, numel, K, count0, er, mode, in_place, fused, seed, keep=None):
    """keep: the intermediate states (1..K-1) the fused forward stores (None:
    all of them); the final state is always stored."""
    hp, _, hm, hv, hc, _, _ = _leaves(numel, seed, True)
    p0 = _device_tree(hp, mode, seed)
    m0 = _device_tree(hm, mode, seed + 1)
    v0 = _device_tree(hv, mode, seed + 2)
    cot = _device_tree(hc, mode, seed + 3)
    G = _grads(numel, K, mode, seed + 10)
    new = lambda j: _empty_like_tree(p0, mode, seed + 50 + j)  # noqa: E731
    stored = lambda k: keep is None or k in keep or k == K  # noqa: E731
    mu = [m0] + [new(k) if stored(k + 1) else None for k in range(K)]
    nu = [v0] + [new(K + k) if stored(k + 1) else None for k in range(K)]
    pK = p0 if in_place else new(2 * K)
    dg = [new(2 * K + 1 + k) for k in range(K)]
    dm0, dv0 = new(3 * K + 1), new(3 * K + 2)
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
    bad = np.flatnonzero(x != y)
    assert bad.size == 0, "%s: %d of %d differ, first at %d" % (what, bad.size, x.size, bad[0])


@pytest.mark.parametrize("K,count0,er,mode,in_place", [
    (1, 0, 0.0, "separate", False),
    (3, 5, 1e-8, "packed-views", False),
    (8, 0, 0.0, "separate", True),
    (9, 2, 1e-8, "packed-views", True),
    (17, 0, 1e-8, "separate", False),
])
def test_fused_tree_equals_stepwise_bitwise(K, count0, er, mode, in_place):
    import paper_2211_06934_amd as P
    numel = _numel(K + 3)
    table = P.segtable_create(numel)
    got = _run(P, table, numel, K, count0, er, mode, in_place, True, 7)
    ref = _run(P, table, numel, K, count0, er, mode, in_place, False, 7)
    _same(got["pK"], ref["pK"], "p_K")
    for k in range(K):
        _same(got["mu"][k], ref["mu"][k], "mu_%d" % (k + 1))
        _same(got["nu"][k], ref["nu"][k], "nu_%d" % (k + 1))
        _same(got["dg"][k], ref["dg"][k], "dg_%d" % (k + 1))
    _same(got["dm0"], ref["dm0"], "dmu0")
    _same(got["dv0"], ref["dv0"], "dnu0")


@pytest.mark.parametrize("K,count0,er,mode,in_place,keep", [
    (1, 0, 0.0, "separate", False, ()),
    (3, 5, 1e-8, "packed-views", False, ()),
    (8, 0, 0.0, "separate", True, ()),                  # one recomputed run of the maximum length
    (9, 2, 1e-8, "packed-views", True, (8,)),
    (11, 0, 1e-8, "separate", False, (3, 10)),          # state 8 unstored: carried across the launch boundary
    (17, 0, 0.0, "packed-views", False, (2, 9, 16)),
    (20, 1, 1e-8, "separate", True, (1, 2, 3, 10, 17)),  # stored runs and recomputed runs mixed
])
def test_fused_tree_recomputed_trajectory_equals_stored_bitwise(K, count0, er, mode, in_place, keep):
    # unstored intermediate states (NULL trajectory entries) are recomputed by
    # the VJP from the latest stored one; every output and every stored state
    # equals the fully stored fused run bit for bit
    import paper_2211_06934_amd as P
    numel = _numel(K + 5)
    table = P.segtable_create(numel)
    got = _run(P, table, numel, K, count0, er, mode, in_place, True, 9, keep=set(keep))
    ref = _run(P, table, numel, K, count0, er, mode, in_place, True, 9)
    _same(got["pK"], ref["pK"], "p_K")
    for k in range(K):
        if got["mu"][k] is not None:
            _same(got["mu"][k], ref["mu"][k], "mu_%d" % (k + 1))
            _same(got["nu"][k], ref["nu"][k], "nu_%d" % (k + 1))
        _same(got["dg"][k], ref["dg"][k], "dg_%d" % (k + 1))
    _same(got["dm0"], ref["dm0"], "dmu0")
    _same(got["dv0"], ref["dv0"], "dnu0")


def test_fused_tree_recomputed_many_small_full_size():
    # the 20,000-leaf benchmark tree, K = 3, nothing stored between the
    # initial and final states, against the fully stored run, bit for bit;
    # leaves are views at 128-byte aligned starts in one buffer per tree, as
    # separate allocations would be
    import paper_2211_06934_amd as P
    from workloads import WORKLOADS, torch_normal
    w = WORKLOADS["many_small"]()
    K, numel = w.K, w.numels
    starts = np.zeros(len(numel), np.int64)
    starts[1:] = np.cumsum((np.asarray(numel[:-1]) + 31) // 32 * 32)
    span = int(starts[-1] + numel[-1])
    table = P.segtable_create(numel)

    def tree(buf):
        return [buf[s:s + k] for s, k in zip(starts.tolist(), numel)]

    def new(seed=None, std=1.0):
        buf = torch_normal(span, std, seed, "cuda") if seed is not None else torch.empty(span, device="cuda")
        return tree(buf), buf

    p0 = new(1, 0.05)
    G = [new(10 + k, w.grad_std) for k in range(K)]
    cot = new(3)
    zero = tree(torch.zeros(span, device="cuda"))

    def run(keep_all):
        mu = [zero] + [new()[0] if (keep_all or k == K) else None for k in range(1, K + 1)]
        nu = [zero] + [new()[0] if (keep_all or k == K) else None for k in range(1, K + 1)]
        pK, dg, dm0, dv0 = new()[0], [new()[0] for _ in range(K)], new()[0], new()[0]
        mp = [None if t is None else _ptrs(t) for t in mu]
        vp = [None if t is None else _ptrs(t) for t in nu]
        gp = [_ptrs(g[0]) for g in G]
        P.adam_unrolled_fwd_tree(table, _ptrs(p0[0]), gp, mp, vp, _ptrs(pK), w.count0, LR, B1, B2, EPS, w.eps_root)
        P.adam_unrolled_bwd_tree(table, _ptrs(cot[0]), gp, mp, vp, [_ptrs(t) for t in dg], _ptrs(dm0), _ptrs(dv0),
                                 w.count0, LR, B1, B2, EPS, w.eps_root)
        return pK, mu[K], nu[K], dg, dm0, dv0

    got = run(False)
    ref = run(True)
    torch.cuda.synchronize()
    for what, a, b in [("p_K", got[0], ref[0]), ("mu_K", got[1], ref[1]), ("nu_K", got[2], ref[2]),
                       ("dmu0", got[4], ref[4]), ("dnu0", got[5], ref[5])] + \
            [("dg_%d" % (k + 1), got[3][k], ref[3][k]) for k in range(K)]:
        _same(a, b, what)
