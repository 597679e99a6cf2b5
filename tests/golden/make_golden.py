"""Write the oracle regression snapshots in this folder.

Every value in them is written here, by the CPU oracle alone: fp32 inputs drawn
from numpy's PCG64 stream with the seeds below, and the oracle's fp64 outputs.
The paper prints no worked example, so these are no pins of the oracle; they
freeze its present outputs, so that any later change to its arithmetic shows
up as a changed snapshot (regenerate with ``python tests/golden/make_golden.py``
and name, in the commit, the passage that justifies the change).  The GPU
tests also compare the HIP path against them.

Case: a small parameter tree (one empty leaf among five), packed with the
oracle's pack, K = 3 unrolled Adam steps (Sec. 2.1 / Listing 1, Adam as in
Kingma & Ba) forward and VJP, and the results unpacked; once from a fresh
state (count 0, eps_root 0) and once from a warm one (count 5, eps_root 1e-8).
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402

SHAPES = [[2, 3], [3], [0], [1], [4, 2]]
HYPER = dict(lr=1e-3, b1=0.9, b2=0.999, eps=1e-8)
CASES = [dict(name="fresh", seed=11, K=3, count0=0, eps_root=0.0, warm=False),
         dict(name="warm", seed=12, K=3, count0=5, eps_root=1e-8, warm=True)]


def hexes(a):
    return [float(x).hex() for x in np.asarray(a, np.float64).reshape(-1)]


def f32(rng, n, std):
    return (rng.standard_normal(n) * std).astype(np.float32)


def case(c):
    rng = np.random.Generator(np.random.PCG64(c["seed"]))
    numel = [int(np.prod(s)) for s in SHAPES]
    n, K = sum(numel), c["K"]
    leaves_p = [f32(rng, k, 0.05) for k in numel]
    leaves_g = [[f32(rng, k, 0.01) for k in numel] for _ in range(K)]
    cot = [f32(rng, k, 1.0) for k in numel]
    if c["warm"]:
        m0, v0 = f32(rng, n, 1e-3), np.abs(f32(rng, n, 1e-4))
    else:
        m0, v0 = np.zeros(n, np.float32), np.zeros(n, np.float32)
    p_flat = oracle.pack(leaves_p)
    g_flat = np.stack([oracle.pack(lg) for lg in leaves_g]).astype(np.float64)
    cot_flat = oracle.pack(cot).astype(np.float64)
    h = dict(HYPER, eps_root=c["eps_root"])
    pK, mt, vt = oracle.unrolled_fwd(p_flat.astype(np.float64), g_flat, m0.astype(np.float64),
                                     v0.astype(np.float64), c["count0"], **h)
    _, dg, dm0, dv0 = oracle.unrolled_bwd(cot_flat, g_flat, mt, vt, c["count0"], **h)
    shapes = [tuple(s) for s in SHAPES]
    return {
        "name": c["name"], "K": K, "count0": c["count0"], "hyper": h, "shapes": SHAPES,
        "inputs": {"p0_leaves": [hexes(x) for x in leaves_p],
                   "grad_leaves": [[hexes(x) for x in lg] for lg in leaves_g],
                   "cot_pK_leaves": [hexes(x) for x in cot], "mu0": hexes(m0), "nu0": hexes(v0)},
        "expected": {"p0_flat": hexes(p_flat),
                     "pK_leaves": [hexes(x) for x in oracle.unpack(pK, shapes)],
                     "mu_K": hexes(mt[K]), "nu_K": hexes(vt[K]),
                     "dg_leaves": [[hexes(x) for x in oracle.unpack(dg[k], shapes)] for k in range(K)],
                     "dmu0": hexes(dm0), "dnu0": hexes(dv0)},
    }


def main():
    out = {"about": "oracle regression snapshot written by tests/golden/make_golden.py; values are float.hex",
           "cases": [case(c) for c in CASES]}
    with open(os.path.join(HERE, "oracle_tree_adam_k3.json"), "w") as f:
        f.write('{"about": %s,\n "cases": [\n' % json.dumps(out["about"]))
        f.write(",\n".join("  " + json.dumps(c) for c in out["cases"]))
        f.write("\n]}\n")


if __name__ == "__main__":
    main()
