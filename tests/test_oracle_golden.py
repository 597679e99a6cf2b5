"""The oracle still produces its committed snapshot (tests/golden).

The snapshot is no pin of the oracle (the paper prints no worked example; the
pins are in the other oracle tests): it makes any change to the oracle's
arithmetic visible.  The oracle is plain fp64 C compiled without contraction,
so a rerun on another host differs at most by libm's last-bit rounding of
sqrt/pow; the bar is 1e-13 relative to the largest element."""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "oracle_tree_adam_k3.json")


def load_cases():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


def arr(hexes, dtype=np.float64):
    return np.array([float.fromhex(x) for x in hexes], dtype=dtype)


def _close(got, ref, what):
    got, ref = np.asarray(got, np.float64).reshape(-1), np.asarray(ref, np.float64).reshape(-1)
    scale = max(float(np.max(np.abs(ref))) if ref.size else 0.0, 1e-300)
    assert got.shape == ref.shape, what
    assert np.max(np.abs(got - ref), initial=0.0) <= 1e-13 * scale, what


@pytest.mark.parametrize("case", load_cases(), ids=lambda c: c["name"])
def test_oracle_reproduces_snapshot(case):
    K, h = case["K"], case["hyper"]
    shapes = [tuple(s) for s in case["shapes"]]
    inp, exp = case["inputs"], case["expected"]
    leaves_p = [arr(x, np.float32) for x in inp["p0_leaves"]]
    leaves_g = [[arr(x, np.float32) for x in lg] for lg in inp["grad_leaves"]]
    cot = [arr(x, np.float32) for x in inp["cot_pK_leaves"]]
    p_flat = oracle.pack(leaves_p)
    # the pack is a copy: bit for bit
    assert np.array_equal(p_flat.view(np.uint32), arr(exp["p0_flat"], np.float32).view(np.uint32))
    G = np.stack([oracle.pack(lg) for lg in leaves_g]).astype(np.float64)
    pK, mt, vt = oracle.unrolled_fwd(p_flat.astype(np.float64), G, arr(inp["mu0"]), arr(inp["nu0"]),
                                     case["count0"], **h)
    _, dg, dm0, dv0 = oracle.unrolled_bwd(oracle.pack(cot).astype(np.float64), G, mt, vt, case["count0"], **h)
    for j, (got, ref) in enumerate(zip(oracle.unpack(pK, shapes), exp["pK_leaves"])):
        _close(got, arr(ref), "pK leaf %d" % j)
    _close(mt[K], arr(exp["mu_K"]), "mu_K")
    _close(vt[K], arr(exp["nu_K"]), "nu_K")
    for k in range(K):
        for j, (got, ref) in enumerate(zip(oracle.unpack(dg[k], shapes), exp["dg_leaves"][k])):
            _close(got, arr(ref), "dg_%d leaf %d" % (k, j))
    _close(dm0, arr(exp["dmu0"]), "dmu0")
    _close(dv0, arr(exp["dnu0"]), "dnu0")
