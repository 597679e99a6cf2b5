"""Maximum sizes: buffers past 2^31 elements, where any 32-bit element or group
index would wrap.  Each kernel runs at full size on the GPU and is compared
with the oracle (or, for the copies, bit for bit) on sampled elements that
include the first and last ones and those around element 2^31.  About 130 GB
of device memory at most, freed between tests."""
import gc
from types import SimpleNamespace

import numpy as np
import pytest
import torch

import oracle
from tests.support import BWD_RTOL, FWD_RTOL, assert_bits_equal, assert_mag_close, stats
from tests.test_gpu_unrolled import _check_unrolled
from workloads import HYPER, torch_normal

pytestmark = pytest.mark.gpu

LR, B1, B2, EPS = HYPER["lr"], HYPER["b1"], HYPER["b2"], HYPER["eps"]
BIG = (1 << 31) + 7  # ragged: the last 3 elements take the tail path


@pytest.fixture(autouse=True)
def _free_device_memory():
    yield
    gc.collect()
    torch.cuda.empty_cache()


def _index(n, seed, count=4096):
    rng = np.random.default_rng(seed)
    edge = [np.arange(64), np.arange(n - 64, n)]
    if n > (1 << 31) + 64:
        edge.append(np.arange((1 << 31) - 64, (1 << 31) + 64))
    return np.unique(np.concatenate(edge + [rng.integers(0, n, size=count)]))


def _take(t, ti):
    return t.index_select(0, ti).cpu().numpy().astype(np.float64)


def test_fused_unrolled_past_2_31():
    w = SimpleNamespace(K=2, n=BIG, grad_std=1e-3, eps_root=1e-8, count0=0)
    _check_unrolled(w, sample=4096)


def test_single_step_past_2_31():
    import paper_2211_06934_amd as P
    n, count, er = BIG, 100, 1e-8
    p, g, m = (torch_normal(n, s, seed, "cuda") for s, seed in ((0.05, 1), (1e-3, 2), (1e-4, 3)))
    v = torch_normal(n, 1e-4, 4, "cuda").abs_()
    po, mo, vo = (torch.empty(n, device="cuda") for _ in range(3))
    P.adam_fwd(p, g, m, v, count, LR, B1, B2, EPS, er, po, mo, vo)
    torch.cuda.synchronize()
    idx = _index(n, 5)
    ti = torch.from_numpy(idx).cuda()
    hp, hg, hm, hv = (_take(x, ti) for x in (p, g, m, v))
    ref = oracle.adam_fwd(hp, hg, hm, hv, count, LR, B1, B2, EPS, er)
    mag = oracle.adam_fwd_mag(hp, hg, hm, hv, count, LR, B1, B2, EPS, er)
    for got, r, mg, what in zip((po, mo, vo), ref[:3], mag[:3], ("p'", "m'", "v'")):
        assert_mag_close(_take(got, ti), r, mg, FWD_RTOL, what)
    del po, mo, vo
    dP, dM, dV = (torch_normal(n, 1.0, seed, "cuda") for seed in (6, 7, 8))
    dg, dmi, dvi = (torch.empty(n, device="cuda") for _ in range(3))
    P.adam_bwd(dP, dM, dV, g, m, v, count, LR, B1, B2, EPS, er, None, dg, dmi, dvi)
    torch.cuda.synchronize()
    hdP, hdM, hdV = (_take(x, ti) for x in (dP, dM, dV))
    ref = oracle.adam_bwd(hdP, hdM, hdV, hg, hm, hv, count, LR, B1, B2, EPS, er)
    mag = oracle.adam_bwd_mag(hdP, hdM, hdV, hg, hm, hv, count, LR, B1, B2, EPS, er)
    for got, r, mg, what in zip((dg, dmi, dvi), ref[1:], mag, ("dg", "dm", "dv")):
        assert_mag_close(_take(got, ti), r, mg, BWD_RTOL, what)


def test_tree_copy_leaf_past_2_31():
    import paper_2211_06934_amd as P
    numel = [5, (1 << 31) + 3, 7]
    table = P.segtable_create(numel)
    n = int(sum(numel))
    leaves = [torch.empty(k, device="cuda") for k in numel]
    for j, x in enumerate(leaves):  # element i of leaf j holds the 32 low bits of i + j * 0x9E3779B1
        a = torch.arange(x.numel(), device="cuda", dtype=torch.int64).add_(j * 0x9E3779B1).bitwise_and_(0xFFFFFFFF)
        a = torch.where(a >= (1 << 31), a - (1 << 32), a)
        x.view(torch.int32).copy_(a)
        del a
    ptrs = torch.tensor([x.data_ptr() for x in leaves], dtype=torch.int64, device="cuda")
    flat = torch.empty(n, device="cuda")
    P.tree_flatten(table, ptrs, flat)
    out = [torch.empty(k, device="cuda") for k in numel]
    optrs = torch.tensor([x.data_ptr() for x in out], dtype=torch.int64, device="cuda")
    P.tree_unflatten(table, flat, optrs)
    torch.cuda.synchronize()
    big = numel[1]
    idx = _index(big, 9)
    ti = torch.from_numpy(idx).cuda()

    def pattern(i, j):
        return ((np.asarray(i, np.int64) + j * 0x9E3779B1) & 0xFFFFFFFF).astype(np.uint32).view(np.int32)

    expect = pattern(idx, 1)
    assert_bits_equal(flat.view(torch.int32).index_select(0, ti + 5).cpu().numpy(), expect, "flat (leaf 1)")
    assert_bits_equal(out[1].view(torch.int32).index_select(0, ti).cpu().numpy(), expect, "unflatten (leaf 1)")
    assert_bits_equal(flat.view(torch.int32)[:5].cpu().numpy(), pattern(np.arange(5), 0), "flat (leaf 0)")
    tail = flat.view(torch.int32)[5 + big:].cpu().numpy()
    assert_bits_equal(tail, pattern(np.arange(7), 2), "flat (leaf 2)")
    assert_bits_equal(out[2].view(torch.int32).cpu().numpy(), tail, "unflatten (leaf 2)")
    assert_bits_equal(out[0].view(torch.int32).cpu().numpy(), pattern(np.arange(5), 0), "unflatten (leaf 0)")


def test_leaf_direct_fused_leaf_past_2_31():
    import paper_2211_06934_amd as P
    numel = [3, (1 << 31) + 5]
    table = P.segtable_create(numel)
    K, er = 2, 0.0

    def tree(std=None, seed=0, zero=False):
        if zero:
            return [torch.zeros(k, device="cuda") for k in numel]
        if std is None:
            return [torch.empty(k, device="cuda") for k in numel]
        return [torch_normal(k, std, seed + j, "cuda") for j, k in enumerate(numel)]

    ptr = lambda t: torch.tensor([x.data_ptr() for x in t], dtype=torch.int64, device="cuda")  # noqa: E731
    p0 = tree(0.05, 10)
    G = [tree(1e-3, 20 + 2 * k) for k in range(K)]
    mu = [tree(zero=True)] + [tree() for _ in range(K)]
    nu = [tree(zero=True)] + [tree() for _ in range(K)]
    pK = tree()
    P.adam_unrolled_fwd_tree(table, ptr(p0), [ptr(t) for t in G], [ptr(t) for t in mu], [ptr(t) for t in nu],
                             ptr(pK), 0, LR, B1, B2, EPS, er)
    cot = tree(1.0, 30)
    dg = [tree() for _ in range(K)]
    dm0, dv0 = tree(), tree()
    P.adam_unrolled_bwd_tree(table, ptr(cot), [ptr(t) for t in G], [ptr(t) for t in mu], [ptr(t) for t in nu],
                             [ptr(t) for t in dg], ptr(dm0), ptr(dv0), 0, LR, B1, B2, EPS, er)
    torch.cuda.synchronize()
    idx = _index(numel[1], 11)
    ti = torch.from_numpy(idx).cuda()
    h = lambda t: _take(t[1], ti)  # noqa: E731
    hG = np.stack([h(t) for t in G])
    z = np.zeros(idx.size)
    pK_ref, mt, vt = oracle.unrolled_fwd(h(p0), hG, z, z, 0, LR, B1, B2, EPS, er)
    mag_p = np.abs(h(p0))
    for k in range(K):
        mag_p = mag_p + oracle.adam_fwd_mag(h(p0), hG[k], mt[k], vt[k], k, LR, B1, B2, EPS, er)[3]
    assert_mag_close(h(pK), pK_ref, mag_p, FWD_RTOL, "p_K")
    for k in range(K):  # each step from the GPU's own state
        hm, hv = h(mu[k]), h(nu[k])
        r = oracle.adam_fwd(h(p0), hG[k], hm, hv, k, LR, B1, B2, EPS, er)
        mg = oracle.adam_fwd_mag(h(p0), hG[k], hm, hv, k, LR, B1, B2, EPS, er)
        assert_mag_close(h(mu[k + 1]), r[1], mg[1], FWD_RTOL, "mu_%d" % (k + 1))
        assert_mag_close(h(nu[k + 1]), r[2], mg[2], FWD_RTOL, "nu_%d" % (k + 1))
    # local backward: the oracle on the GPU's own trajectory, scales carried through the steps
    hmt = np.stack([h(t) for t in mu])
    hvt = np.stack([h(t) for t in nu])
    hcot = h(cot)
    _, dg_ref, dm_ref, dv_ref = oracle.unrolled_bwd(hcot, hG, hmt, hvt, 0, LR, B1, B2, EPS, er)
    magM = np.zeros(idx.size)
    magV = np.zeros(idx.size)
    for k in range(K, 0, -1):
        mg, mm, mv = oracle.adam_bwd_mag(hcot, magM, magV, hG[k - 1], hmt[k - 1], hvt[k - 1], k - 1, LR, B1, B2,
                                         EPS, er)
        assert_mag_close(h(dg[k - 1]), dg_ref[k - 1], mg, BWD_RTOL, "dg_%d" % k)
        magM, magV = mm, mv
    assert_mag_close(h(dm0), dm_ref, magM, BWD_RTOL, "dm0")
    assert_mag_close(h(dv0), dv_ref, magV, BWD_RTOL, "dv0")


def test_es_rows_past_2_31_elements():
    import paper_2211_06934_amd as P
    N, n, sigma = 3, (1 << 30) + 4, 0.05
    theta = torch_normal(n, 1.0, 40, "cuda")
    noise = torch_normal(N * n, 1.0, 41, "cuda").reshape(N, n)
    out = torch.empty(2 * N, n, device="cuda")
    P.es_perturb(theta, noise, sigma, True, out)
    w = torch.tensor([0.5, -1.25, 2.0], device="cuda")
    g = torch.empty(n, device="cuda")
    P.es_estimate(noise, w, 1.0 / (2 * N * sigma), g)
    torch.cuda.synchronize()
    idx = np.unique(np.concatenate([np.arange(64), np.arange(n - 64, n),
                                    np.random.default_rng(12).integers(0, n, 4096)]))
    ti = torch.from_numpy(idx).cuda()
    ht = _take(theta, ti)
    hz = np.stack([_take(noise[i], ti) for i in range(N)])
    ref = oracle.es_perturb(ht, hz, sigma, True)
    got = np.stack([_take(out[i], ti) for i in range(2 * N)])
    mag = np.abs(ht)[None, :] + sigma * np.abs(np.concatenate([hz, hz]))
    assert_mag_close(got, ref, mag, FWD_RTOL, "perturb")
    hw = w.cpu().numpy().astype(np.float64)
    scale = 1.0 / (2 * N * sigma)
    assert_mag_close(_take(g, ti), oracle.es_estimate(hz, hw, scale), oracle.es_estimate_mag(hz, hw, scale),
                     BWD_RTOL, "estimate")


@pytest.mark.parametrize("n", [(1 << 31) + 8, BIG])
def test_es_gaussian_past_2_31(n):
    """In-kernel noise at a parameter count past 2^31 (n = 2^31 + 8 takes the
    128-bit path, 2^31 + 7 the scalar one): perturbation and estimate on
    sampled parameters against the oracle's noise for those columns."""
    import paper_2211_06934_amd as P
    N, sigma, seed = 2, 0.05, 0xB16B00B5
    theta = torch_normal(n, 1.0, 42, "cuda")
    out = torch.empty(2 * N, n, device="cuda")
    P.es_perturb_gaussian(theta, N, seed, sigma, True, out)
    f = torch.tensor([1.5, -0.25, 0.75, 2.0], device="cuda")
    g = torch.empty(n, device="cuda")
    P.es_estimate_gaussian(f, "antithetic", N, seed, sigma, g)
    torch.cuda.synchronize()
    idx = _index(n, 13)
    ti = torch.from_numpy(idx).cuda()
    ht = _take(theta, ti)
    z, r = oracle.es_gaussian_noise_cols(N, idx, seed)
    got = np.stack([_take(out[i], ti) for i in range(2 * N)])
    mag = np.abs(ht)[None, :] + sigma * np.concatenate([r, r])
    assert_mag_close(got, oracle.es_perturb(ht, z, sigma, True), mag, FWD_RTOL, "perturb")
    hf = f.cpu().numpy()
    w, scale = oracle.es_weights(hf, "antithetic", sigma)
    mag = oracle.es_estimate_mag(r, oracle.es_weight_terms(hf, "antithetic"), scale)
    assert_mag_close(_take(g, ti), oracle.es_estimate(z, w, scale), mag, BWD_RTOL, "estimate")


def _end_to_end(h_p0, hG, h_cot, got_pK, got_muK, got_nuK, got_dg, got_dm0, got_dv0, er):
    """Against the all-fp64 oracle from the same fp32 inputs on the sampled
    elements: p_K within FWD_RTOL of its summed scales, the final moments and
    the meta-gradients norm-relative (the end-to-end bars of the parity tests)."""
    K = hG.shape[0]
    z = np.zeros(h_p0.size)
    pK_ref, mt, vt = oracle.unrolled_fwd(h_p0, hG, z, z, 0, LR, B1, B2, EPS, er)
    mag_p = np.abs(h_p0)
    for k in range(K):
        mag_p = mag_p + oracle.adam_fwd_mag(h_p0, hG[k], mt[k], vt[k], k, LR, B1, B2, EPS, er)[3]
    assert_mag_close(got_pK, pK_ref, mag_p, FWD_RTOL, "p_K")
    assert stats(got_muK, mt[K])[1] < FWD_RTOL and stats(got_nuK, vt[K])[1] < FWD_RTOL
    _, dg_r, dm_r, dv_r = oracle.unrolled_bwd(h_cot, hG, mt, vt, 0, LR, B1, B2, EPS, er)
    worst = max([stats(got_dg[k], dg_r[k])[1] for k in range(K)] + [stats(got_dm0, dm_r)[1],
                                                                     stats(got_dv0, dv_r)[1]])
    assert worst < BWD_RTOL, worst


def test_recomputed_trajectory_past_2_31():
    # flat K-step driver with nothing stored between the initial and final
    # states: the VJP recomputes the moments (the benchmark's policy)
    import paper_2211_06934_amd as P
    n, K, er = BIG, 3, 1e-8
    p0 = torch_normal(n, 0.05, 50, "cuda")
    G = [torch_normal(n, 1e-3, 51 + k, "cuda") for k in range(K)]
    mt = [torch.zeros(n, device="cuda")] + [None] * (K - 1) + [torch.empty(n, device="cuda")]
    vt = [torch.zeros(n, device="cuda")] + [None] * (K - 1) + [torch.empty(n, device="cuda")]
    pK = torch.empty(n, device="cuda")
    P.adam_unrolled_fwd(p0, G, mt, vt, pK, 0, LR, B1, B2, EPS, er)
    cot = torch_normal(n, 1.0, 55, "cuda")
    dg = [torch.empty(n, device="cuda") for _ in range(K)]
    dm0, dv0 = torch.empty(n, device="cuda"), torch.empty(n, device="cuda")
    P.adam_unrolled_bwd(cot, G, mt, vt, dg, dm0, dv0, 0, LR, B1, B2, EPS, er)
    torch.cuda.synchronize()
    ti = torch.from_numpy(_index(n, 13)).cuda()
    _end_to_end(_take(p0, ti), np.stack([_take(x, ti) for x in G]), _take(cot, ti), _take(pK, ti),
                _take(mt[K], ti), _take(vt[K], ti), [_take(x, ti) for x in dg], _take(dm0, ti), _take(dv0, ti), er)


def test_leaf_direct_recomputed_trajectory_past_2_31():
    import paper_2211_06934_amd as P
    numel = [3, (1 << 31) + 5]
    table = P.segtable_create(numel)
    K, er = 3, 0.0

    def tree(std=None, seed=0, zero=False):
        if zero:
            return [torch.zeros(k, device="cuda") for k in numel]
        if std is None:
            return [torch.empty(k, device="cuda") for k in numel]
        return [torch_normal(k, std, seed + j, "cuda") for j, k in enumerate(numel)]

    ptr = lambda t: torch.tensor([x.data_ptr() for x in t], dtype=torch.int64, device="cuda")  # noqa: E731
    p0 = tree(0.05, 60)
    G = [tree(1e-3, 62 + 2 * k) for k in range(K)]
    mu0, nu0, muK, nuK = tree(zero=True), tree(zero=True), tree(), tree()  # held: the VJP reads mu0, nu0
    mu = [ptr(mu0)] + [None] * (K - 1) + [ptr(muK)]
    nu = [ptr(nu0)] + [None] * (K - 1) + [ptr(nuK)]
    pK = tree()
    P.adam_unrolled_fwd_tree(table, ptr(p0), [ptr(t) for t in G], mu, nu, ptr(pK), 0, LR, B1, B2, EPS, er)
    cot = tree(1.0, 70)
    dg = [tree() for _ in range(K)]
    dm0, dv0 = tree(), tree()
    P.adam_unrolled_bwd_tree(table, ptr(cot), [ptr(t) for t in G], mu, nu, [ptr(t) for t in dg], ptr(dm0),
                             ptr(dv0), 0, LR, B1, B2, EPS, er)
    torch.cuda.synchronize()
    ti = torch.from_numpy(_index(numel[1], 17)).cuda()
    h = lambda t: _take(t[1], ti)  # noqa: E731
    _end_to_end(h(p0), np.stack([h(t) for t in G]), h(cot), h(pK), h(muK), h(nuK), [h(t) for t in dg], h(dm0),
                h(dv0), er)
