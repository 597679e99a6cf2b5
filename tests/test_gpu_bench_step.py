"""The benchmark's own timed steps (every workload it offers but the flat 10^9
cases, which tests/test_gpu_unrolled.py covers in their own launch
configuration, and the torch comparison), at full size, against the oracle.

bench.py's setup and step functions are called as they are (same leaves,
same batched copies, same store policy and launch plan), and the outputs are
compared with the oracle on a seeded sample of elements: every operation on
the path is elementwise (the copies move each element on its own), so the
oracle computes any sampled element from that element's inputs alone.

  - pack and unpack: the flat buffers equal the concatenated leaves bit for
    bit (checked in full on the device);
  - forward: p_K per element within 1e-5 of its term scale, propagated over
    the K steps of the all-fp64 run; the final moments norm-relative 1e-5;
  - VJP: every dg_k, dmu0, dnu0 against the all-fp64 oracle from the same
    fp32 inputs, norm-relative 1e-4 (the moment trajectory is recomputed on
    the GPU, so the end-to-end reading applies).
"""
import importlib.util
import os

import numpy as np
import pytest
import torch

import oracle
from tests.support import BWD_RTOL, FWD_RTOL, assert_mag_close, stats
from workloads import WORKLOADS

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _sample(n, count, seed):
    rng = np.random.default_rng(seed)
    idx = np.concatenate([np.arange(min(n, 1024)), np.arange(max(0, n - 1024), n), rng.integers(0, n, size=count)])
    return torch.from_numpy(np.unique(idx)).cuda()


def _cat(leaves):
    return torch.cat([x.reshape(-1) for x in leaves])


def _check_adam(S, flat, idx):
    """flat: dict of full-size flat device buffers p0, g (list), cot, pK, muK,
    nuK, dg (list), dm0, dv0 as the step left them."""
    K, h = S["K"], S["hyper"]
    hp = (h["lr"], h["b1"], h["b2"], h["eps"], h["eps_root"])
    at = lambda t: t.index_select(0, idx).cpu().numpy().astype(np.float64)  # noqa: E731
    p0, cot = at(flat["p0"]), at(flat["cot"])
    G = np.stack([at(g) for g in flat["g"]])
    z = np.zeros_like(p0)
    pK_ref, mt_ref, vt_ref = oracle.unrolled_fwd(p0, G, z, z, S["count0"], *hp)
    mag_p = np.abs(p0)
    for k in range(1, K + 1):
        mag_p = mag_p + oracle.adam_fwd_mag(p0, G[k - 1], mt_ref[k - 1], vt_ref[k - 1], S["count0"] + k - 1, *hp)[3]
    assert_mag_close(at(flat["pK"]), pK_ref, mag_p, FWD_RTOL, "p_K")
    assert stats(at(flat["muK"]), mt_ref[K])[1] < FWD_RTOL, "mu_K"
    assert stats(at(flat["nuK"]), vt_ref[K])[1] < FWD_RTOL, "nu_K"
    _, dg_r, dm0_r, dv0_r = oracle.unrolled_bwd(cot, G, mt_ref, vt_ref, S["count0"], *hp)
    for k in range(K):
        assert stats(at(flat["dg"][k]), dg_r[k])[1] < BWD_RTOL, "dg_%d" % k
    assert stats(at(flat["dm0"]), dm0_r)[1] < BWD_RTOL, "dmu0"
    assert stats(at(flat["dv0"]), dv0_r)[1] < BWD_RTOL, "dnu0"


@pytest.mark.parametrize("name", ["many_small", "resnet18_k10", "resnet18_k1", "convnet32", "tiny_mlp"])
def test_flatten_fused_unflatten_step(name):
    import paper_2211_06934_amd as P
    b = _bench()
    w = WORKLOADS[name]()
    S = b.setup_tree(torch, P, w, "recompute")
    b.step_tree(P, S)
    torch.cuda.synchronize()
    p_tree, g_trees, pK_tree, dg_trees = S["keep"]
    K = S["K"]
    # the copies: flat inputs are the packed leaves, unpacked outputs the flat results
    assert torch.equal(S["p0"].view(torch.int32), _cat(p_tree).view(torch.int32))
    for k in range(K):
        assert torch.equal(S["g"][k].view(torch.int32), _cat(g_trees[k]).view(torch.int32)), k
        assert torch.equal(S["dg"][k].view(torch.int32), _cat(dg_trees[k]).view(torch.int32)), k
    assert torch.equal(S["pK"].view(torch.int32), _cat(pK_tree).view(torch.int32))
    flat = dict(p0=S["p0"], g=S["g"], cot=S["cot"], pK=S["pK"], muK=S["mu"][K], nuK=S["nu"][K], dg=S["dg"],
                dm0=S["dm0"], dv0=S["dv0"])
    _check_adam(S, flat, _sample(S["n"], 200_000, 11))


def test_leaf_direct_step():
    import paper_2211_06934_amd as P
    b = _bench()
    S = b.setup_treemap(torch, P, WORKLOADS["many_small"](), "recompute")
    b.step_treemap(P, S)
    torch.cuda.synchronize()
    n, K = S["n"], S["K"]

    def flat(ptrs):
        out = torch.empty(n, device="cuda")
        P.tree_flatten(S["table"], ptrs, out)
        return out

    fl = dict(p0=flat(S["p0"]), g=[flat(g) for g in S["g"]], cot=flat(S["cot"]), pK=flat(S["pK"]),
              muK=flat(S["mu"][K]), nuK=flat(S["nu"][K]), dg=[flat(d) for d in S["dg"]], dm0=flat(S["dm0"]),
              dv0=flat(S["dv0"]))
    torch.cuda.synchronize()
    _check_adam(S, fl, _sample(n, 200_000, 12))


@pytest.mark.parametrize("which", ["sgd", "rmsprop"])
def test_leaf_direct_sgd_rmsprop_step(which):
    import paper_2211_06934_amd as P
    b = _bench()
    S = b.setup_optim_tree(torch, P, which, WORKLOADS["many_small"]())
    b.step_optim_tree(P, S)
    torch.cuda.synchronize()
    n = S["n"]
    idx = _sample(n, 200_000, 13)

    def at(ptrs):
        out = torch.empty(n, device="cuda")
        P.tree_flatten(S["table"], ptrs, out)
        return out.index_select(0, idx).cpu().numpy().astype(np.float64)

    p, g, dP = at(S["p"]), at(S["g"]), at(S["dP"])
    if which == "sgd":
        t, dT = at(S["t"]), at(S["dT"])
        ref = oracle.sgd_fwd(p, g, t, S["lr"], S["mom"], True)
        mag = oracle.sgd_fwd_mag(p, g, t, S["lr"], S["mom"], True)
        for got, r, m, what in zip((at(S["po"]), at(S["to"])), ref, mag, ("p'", "t'")):
            assert_mag_close(got, r, m, FWD_RTOL, what)
        ref = oracle.sgd_bwd(dP, dT, S["lr"], S["mom"], True)[1:]  # (dg, dt)
        mag = oracle.sgd_bwd_mag(dP, dT, S["lr"], S["mom"], True)
        for got, r, m, what in zip((at(S["dg"]), at(S["dt"])), ref, mag, ("dg", "dt")):
            assert_mag_close(got, r, m, BWD_RTOL, what)
    else:
        v, bb, dV, dB = at(S["v"]), at(S["b"]), at(S["dV"]), at(S["dB"])
        hp = (S["lr"], 0.99, 1e-8, 0.0, S["mom"])
        ref = oracle.rmsprop_fwd(p, g, v, bb, *hp)
        mag = oracle.rmsprop_fwd_mag(p, g, v, bb, *hp)
        for got, r, m, what in zip((at(S["po"]), at(S["vo"]), at(S["bo"])), ref, mag, ("p'", "v'", "b'")):
            assert_mag_close(got, r, m, FWD_RTOL, what)
        ref = oracle.rmsprop_bwd(dP, dV, dB, g, v, *hp)[1:]  # (dg, dv, db)
        mag = oracle.rmsprop_bwd_mag(dP, dV, dB, g, v, *hp)
        for got, r, m, what in zip((at(S["dg"]), at(S["dv"]), at(S["db"])), ref, mag, ("dg", "dv", "db")):
            assert_mag_close(got, r, m, BWD_RTOL, what)


@pytest.mark.parametrize("which", ["sgd", "rmsprop"])
def test_flat_sgd_rmsprop_step(which):
    import paper_2211_06934_amd as P
    b = _bench()
    S = b.setup_optim(torch, P, which)
    b.step_optim(P, S)
    torch.cuda.synchronize()
    idx = _sample(S["n"], 200_000, 14)
    at = lambda t: t.index_select(0, idx).cpu().numpy().astype(np.float64)  # noqa: E731
    p, g, dP = at(S["p"]), at(S["g"]), at(S["dP"])
    if which == "sgd":
        t, dT = at(S["t"]), at(S["dT"])
        fwd = zip((at(S["po"]), at(S["to"])), oracle.sgd_fwd(p, g, t, S["lr"], S["mom"], True),
                  oracle.sgd_fwd_mag(p, g, t, S["lr"], S["mom"], True))
        bwd = zip((at(S["dg"]), at(S["dt"])), oracle.sgd_bwd(dP, dT, S["lr"], S["mom"], True)[1:],
                  oracle.sgd_bwd_mag(dP, dT, S["lr"], S["mom"], True))
    else:
        v, bb, dV, dB = at(S["v"]), at(S["b"]), at(S["dV"]), at(S["dB"])
        hp = (S["lr"], 0.99, 1e-8, 0.0, S["mom"])
        fwd = zip((at(S["po"]), at(S["vo"]), at(S["bo"])), oracle.rmsprop_fwd(p, g, v, bb, *hp),
                  oracle.rmsprop_fwd_mag(p, g, v, bb, *hp))
        bwd = zip((at(S["dg"]), at(S["dv"]), at(S["db"])), oracle.rmsprop_bwd(dP, dV, dB, g, v, *hp)[1:],
                  oracle.rmsprop_bwd_mag(dP, dV, dB, g, v, *hp))
    for i, (got, r, m) in enumerate(fwd):
        assert_mag_close(got, r, m, FWD_RTOL, "fwd output %d" % i)
    for i, (got, r, m) in enumerate(bwd):
        assert_mag_close(got, r, m, BWD_RTOL, "bwd output %d" % i)


@pytest.mark.parametrize("noise_input", [False, True])
def test_es_step(noise_input):
    # ResNet-18 size, 64 antithetic rows: sampled columns of the points and
    # of the estimate (every column is computed from its own column of noise:
    # regenerated by the oracle from the seed, or read from the noise array)
    import paper_2211_06934_amd as P
    b = _bench()
    S = b.setup_es(torch, P, WORKLOADS["resnet18_k1"](), noise_input)
    b.step_es(P, S)
    torch.cuda.synchronize()
    idx = _sample(S["n"], 50_000, 15)
    cols = lambda t: t.index_select(1, idx).cpu().numpy().astype(np.float64)  # noqa: E731
    theta = S["theta"].index_select(0, idx).cpu().numpy().astype(np.float64)
    sigma, N = S["sigma"], S["N"]
    if noise_input:
        Z = cols(S["noise"])
        R = np.abs(Z)
    else:
        Z, R = oracle.es_gaussian_noise_cols(N, idx.cpu().numpy(), S["seed"])
    mag = np.abs(theta)[None, :] + sigma * np.concatenate([R, R])
    assert_mag_close(cols(S["pts"]), oracle.es_perturb(theta, Z, sigma, True), mag, FWD_RTOL, "perturb")
    f = S["fvals"].cpu().numpy().astype(np.float64)
    w, scale = oracle.es_weights(f, "antithetic", sigma)
    terms = oracle.es_weight_terms(f, "antithetic")
    g = S["grad"].index_select(0, idx).cpu().numpy().astype(np.float64)
    assert_mag_close(g, oracle.es_estimate(Z, w, scale), oracle.es_estimate_mag(R, terms, scale), BWD_RTOL,
                     "estimate")


def test_stepwise_pass():
    # the one-launch-per-step form of the default pass: the same outputs as
    # the oracle, and bit for bit those of the fused driver on the same inputs
    import paper_2211_06934_amd as P
    b = _bench()
    w = WORKLOADS["many_small"]()
    S = b.setup_stepwise(torch, P, w)
    b.step_stepwise(P, S)
    torch.cuda.synchronize()
    K = S["K"]
    p_tree, g_trees, pK_tree, dg_trees = S["keep"]
    assert torch.equal(S["pK"].view(torch.int32), _cat(pK_tree).view(torch.int32))
    flat = dict(p0=S["p0"], g=S["g"], cot=S["cot"], pK=S["pK"], muK=S["mu"][K], nuK=S["nu"][K], dg=S["dg"],
                dm0=S["dm0"], dv0=S["dv0"])
    _check_adam(S, flat, _sample(S["n"], 200_000, 16))
    # the fused driver from the same packed inputs
    e = lambda: torch.empty_like(S["p0"])  # noqa: E731
    mt = [S["mu"][0]] + [None] * (K - 1) + [e()]
    vt = [S["nu"][0]] + [None] * (K - 1) + [e()]
    pK, dg, dm0, dv0 = e(), [e() for _ in range(K)], e(), e()
    h = S["hyper"]
    co = (S["count0"], h["lr"], h["b1"], h["b2"], h["eps"], h["eps_root"])
    P.adam_unrolled_fwd(S["p0"], S["g"], mt, vt, pK, *co)
    P.adam_unrolled_bwd(S["cot"], S["g"], mt, vt, dg, dm0, dv0, *co)
    torch.cuda.synchronize()
    pairs = [(pK, S["pK"]), (mt[K], S["mu"][K]), (vt[K], S["nu"][K]), (dm0, S["dm0"]), (dv0, S["dv0"])]
    for a, c in pairs + list(zip(dg, S["dg"])):
        assert torch.equal(a.view(torch.int32), c.view(torch.int32))


@pytest.mark.parametrize("name", ["tiny_mlp", "convnet32", "resnet18_k1", "resnet18_k10"])
def test_small_tree_forms_agree_bit_for_bit(name):
    # the three forms the small-trees benchmark times -- pack + fused K-step +
    # unpack, leaf-direct fused K-step, leaf-direct one launch per step --
    # compute every element with the same operations, so p_K, every dg_k and
    # the initial-state cotangents agree bit for bit
    import paper_2211_06934_amd as P
    b = _bench()
    w = WORKLOADS[name]()
    A = b.setup_tree(torch, P, w, "recompute")
    b.step_tree(P, A)
    K, n = A["K"], A["n"]
    ref = [A["pK"]] + A["dg"] + [A["dm0"], A["dv0"]]
    for stepwise in (False, True):
        S = b.setup_treemap(torch, P, w, "stored" if stepwise else "recompute", stepwise=stepwise)
        (b.step_treemap_stepwise if stepwise else b.step_treemap)(P, S)

        def flat(ptrs):
            out = torch.empty(n, device="cuda")
            P.tree_flatten(S["table"], ptrs, out)
            return out

        got = [flat(S["pK"])] + [flat(d) for d in S["dg"]] + [flat(S["dm0"]), flat(S["dv0"])]
        torch.cuda.synchronize()
        for i, (x, y) in enumerate(zip(got, ref)):
            assert torch.equal(x.view(torch.int32), y.view(torch.int32)), (name, stepwise, i)
    assert K == len(A["dg"])
