"""GPU parity of the K-step unrolled driver (Listing 1's loop and its
meta-gradient) on the workload trees, and of one interior fwd+bwd step on the
flat 1B-parameter buffer, against the oracle.

Three checks per run:
  local forward   each step's (m_k, v_k) against the oracle step applied to the
                  GPU's own (m_{k-1}, v_{k-1}); p_K against the fp64 run;
  local backward  the oracle's K-step backward on the GPU's saved trajectory,
                  element by element, with tolerance scales propagated through
                  the K steps;
  end to end      the meta-gradients against an all-fp64 oracle run from the
                  same fp32 inputs, norm-relative.
Large workloads run at full size on the GPU and are compared on a seeded
sample of elements (the K-step map is elementwise, so the oracle can compute
any element on its own).
"""
import numpy as np
import pytest
import torch

import oracle
from tests.support import BWD_RTOL, FWD_RTOL, assert_mag_close, stats
from workloads import HYPER, WORKLOADS, host_inputs, torch_normal

pytestmark = pytest.mark.gpu

LR, B1, B2, EPS = HYPER["lr"], HYPER["b1"], HYPER["b2"], HYPER["eps"]


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _sample_index(n, count, seed):
    if n <= count:
        return np.arange(n)
    rng = np.random.default_rng(seed)
    idx = np.concatenate([np.arange(2048), np.arange(n - 2048, n), rng.integers(0, n, size=count)])
    return np.unique(idx)


def _check_unrolled(w, sample=None):
    import paper_2211_06934_amd as P
    K = w.K
    n = w.n
    if sample is None:
        inp = host_inputs(w)
        p0, grads, m0, v0, cot = map(_dev, (inp.p0, inp.grads.reshape(K, n), inp.m0, inp.v0, inp.cot_p))
        gl = [grads[k] for k in range(K)]
    else:
        # draw on the device (too large for a quick host draw), copy samples back
        p0 = torch_normal(n, 0.05, 1, "cuda")
        gl = [torch_normal(n, w.grad_std, 10 + k, "cuda") for k in range(K)]
        m0 = torch.zeros(n, device="cuda")
        v0 = torch.zeros(n, device="cuda")
        cot = torch_normal(n, 1.0, 3, "cuda")
    er = w.eps_root
    mt = [m0] + [torch.empty(n, device="cuda") for _ in range(K)]
    vt = [v0] + [torch.empty(n, device="cuda") for _ in range(K)]
    pK = torch.empty(n, device="cuda")
    P.adam_unrolled_fwd(p0, gl, mt, vt, pK, w.count0, LR, B1, B2, EPS, er)
    dg = [torch.empty(n, device="cuda") for _ in range(K)]
    dm0 = torch.empty(n, device="cuda")
    dv0 = torch.empty(n, device="cuda")
    P.adam_unrolled_bwd(cot, gl, mt, vt, dg, dm0, dv0, w.count0, LR, B1, B2, EPS, er)
    torch.cuda.synchronize()

    idx = _sample_index(n, sample, 7) if sample is not None else None
    ti = None if idx is None else torch.from_numpy(idx).cuda()

    def h(t):
        t = t if ti is None else t.index_select(0, ti)
        return t.cpu().numpy().astype(np.float64)

    hp0, hcot, hm0, hv0 = h(p0), h(cot), h(m0), h(v0)
    hg = np.stack([h(x) for x in gl])
    hmt = np.stack([h(x) for x in mt])
    hvt = np.stack([h(x) for x in vt])

    # local forward: each step from the GPU's own state
    for k in range(1, K + 1):
        ref = oracle.adam_fwd(hp0, hg[k - 1], hmt[k - 1], hvt[k - 1], w.count0 + k - 1, LR, B1, B2, EPS, er)
        mag = oracle.adam_fwd_mag(hp0, hg[k - 1], hmt[k - 1], hvt[k - 1], w.count0 + k - 1, LR, B1, B2, EPS, er)
        assert_mag_close(hmt[k], ref[1], mag[1], FWD_RTOL, "m_%d" % k)
        assert_mag_close(hvt[k], ref[2], mag[2], FWD_RTOL, "v_%d" % k)
    # p_K against the all-fp64 run; scale |p0| + sum of the steps' update scales
    pK_ref, mt_ref, vt_ref = oracle.unrolled_fwd(hp0, hg, hm0, hv0, w.count0, LR, B1, B2, EPS, er)
    mag_p = np.abs(hp0)
    for k in range(1, K + 1):
        mag_p = mag_p + oracle.adam_fwd_mag(hp0, hg[k - 1], mt_ref[k - 1], vt_ref[k - 1], w.count0 + k - 1,
                                            LR, B1, B2, EPS, er)[3]
    assert_mag_close(h(pK), pK_ref, mag_p, FWD_RTOL, "p_K")

    # local backward: oracle on the GPU's trajectory, scales carried through the steps
    dp0_l, dg_l, dm0_l, dv0_l = oracle.unrolled_bwd(hcot, hg, hmt, hvt, w.count0, LR, B1, B2, EPS, er)
    magM = np.zeros_like(hcot)
    magV = np.zeros_like(hcot)
    for k in range(K, 0, -1):
        mg, mm, mv = oracle.adam_bwd_mag(hcot, magM, magV, hg[k - 1], hmt[k - 1], hvt[k - 1], w.count0 + k - 1,
                                         LR, B1, B2, EPS, er)
        assert_mag_close(h(dg[k - 1]), dg_l[k - 1], mg, BWD_RTOL, "dg_%d" % k)
        magM, magV = mm, mv
    assert_mag_close(h(dm0), dm0_l, magM, BWD_RTOL, "dm0")
    assert_mag_close(h(dv0), dv0_l, magV, BWD_RTOL, "dv0")

    # end to end: all-fp64 oracle from the fp32 inputs, norm-relative
    _, dg_r, dm0_r, dv0_r = oracle.unrolled_bwd(hcot, hg, mt_ref, vt_ref, w.count0, LR, B1, B2, EPS, er)
    worst = 0.0
    for k in range(K):
        worst = max(worst, stats(h(dg[k]), dg_r[k])[1])
    worst = max(worst, stats(h(dm0), dm0_r)[1], stats(h(dv0), dv0_r)[1])
    assert worst < BWD_RTOL, worst
    return worst


@pytest.mark.parametrize("name", ["tiny_mlp", "convnet32", "resnet18_k1"])
def test_unrolled_full_compare(name):
    _check_unrolled(WORKLOADS[name]())


@pytest.mark.parametrize("name", ["resnet18_k10", "many_small"])
def test_unrolled_full_size_sampled(name):
    _check_unrolled(WORKLOADS[name](), sample=400_000)


def test_unrolled_meta_gradient_vs_fd_of_gpu_forward():
    # The GPU meta-gradient on the tiny tree against central differences of the
    # oracle's K-step forward (fp64), as a direct pin of what the backward means.
    import paper_2211_06934_amd as P
    w = WORKLOADS["tiny_mlp"]()
    K, n = w.K, w.n
    inp = host_inputs(w)
    p0, m0, v0, cot = map(_dev, (inp.p0, inp.m0, inp.v0, inp.cot_p))
    gl = [_dev(inp.grads[k]) for k in range(K)]
    mt = [m0] + [torch.empty(n, device="cuda") for _ in range(K)]
    vt = [v0] + [torch.empty(n, device="cuda") for _ in range(K)]
    pK = torch.empty(n, device="cuda")
    P.adam_unrolled_fwd(p0, gl, mt, vt, pK, 0, LR, B1, B2, EPS, 0.0)
    dg = [torch.empty(n, device="cuda") for _ in range(K)]
    dm0, dv0 = torch.empty(n, device="cuda"), torch.empty(n, device="cuda")
    P.adam_unrolled_bwd(cot, gl, mt, vt, dg, dm0, dv0, 0, LR, B1, B2, EPS, 0.0)
    torch.cuda.synchronize()
    G = inp.grads.astype(np.float64)
    c = inp.cot_p.astype(np.float64)
    z = np.zeros(n)
    for k in range(K):
        rms = float(np.sqrt(np.mean(G[k] ** 2)))
        hstep = 1e-5 * np.maximum(np.abs(G[k]), 1e-2 * rms)
        gp, gm = G.copy(), G.copy()
        gp[k] += hstep
        gm[k] -= hstep
        fd = c * (oracle.unrolled_fwd(inp.p0, gp, z, z, 0, LR, B1, B2, EPS, 0.0)[0] -
                  oracle.unrolled_fwd(inp.p0, gm, z, z, 0, LR, B1, B2, EPS, 0.0)[0]) / (2 * hstep)
        got = dg[k].cpu().numpy().astype(np.float64)
        _, normrel = stats(got, fd)
        assert normrel < BWD_RTOL, (k, normrel)


def test_flat_1b_interior_step_sampled():
    # The flat 1B workload: one fwd with nonzero moments at count 100, then one
    # bwd with all three cotangents nonzero, at full size, in the launch
    # configuration the benchmark times; compared on a seeded sample.
    import paper_2211_06934_amd as P
    w = WORKLOADS["flat_1b"]()
    n = w.n
    print("flat_1b: allocating 13 x %d fp32" % n, flush=True)
    p = torch_normal(n, 0.05, 21, "cuda")
    g = torch_normal(n, w.grad_std, 22, "cuda")
    m = torch_normal(n, 1e-4, 23, "cuda").abs_()
    v = torch_normal(n, 1e-4, 24, "cuda").abs_()
    po, mo, vo = (torch.empty(n, device="cuda") for _ in range(3))
    P.adam_fwd(p, g, m, v, w.count0, LR, B1, B2, EPS, w.eps_root, po, mo, vo)
    dP = torch_normal(n, 1.0, 25, "cuda")
    dM = torch_normal(n, 1.0, 26, "cuda")
    dV = torch_normal(n, 1.0, 27, "cuda")
    dg, dm, dv = (torch.empty(n, device="cuda") for _ in range(3))
    P.adam_bwd(dP, dM, dV, g, m, v, w.count0, LR, B1, B2, EPS, w.eps_root, None, dg, dm, dv)
    torch.cuda.synchronize()
    idx = torch.from_numpy(_sample_index(n, 1_000_000, 3)).cuda()

    def h(t):
        return t.index_select(0, idx).cpu().numpy().astype(np.float64)

    hp, hg, hm, hv, hP, hM, hV = map(h, (p, g, m, v, dP, dM, dV))
    ref = oracle.adam_fwd(hp, hg, hm, hv, w.count0, LR, B1, B2, EPS, w.eps_root)
    mag = oracle.adam_fwd_mag(hp, hg, hm, hv, w.count0, LR, B1, B2, EPS, w.eps_root)
    for name, got, r, mg in zip(("p'", "m'", "v'"), (h(po), h(mo), h(vo)), ref, mag):
        assert_mag_close(got, r, mg, FWD_RTOL, name)
    refb = oracle.adam_bwd(hP, hM, hV, hg, hm, hv, w.count0, LR, B1, B2, EPS, w.eps_root)
    magb = oracle.adam_bwd_mag(hP, hM, hV, hg, hm, hv, w.count0, LR, B1, B2, EPS, w.eps_root)
    for name, got, r, mg in zip(("dg", "dm", "dv"), (h(dg), h(dm), h(dv)), refb[1:], magb):
        assert_mag_close(got, r, mg, BWD_RTOL, name)
