"""Randomized check of the leaf-direct single-step Adam forward and VJP: on
seeded random tables (empty, tiny and large leaves; separate leaves or views
at random phases inside one buffer; with and without moment cotangents) the
leaf-direct results equal the flat kernels' on the concatenated leaves bit
for bit.  The flat kernels are held to the oracle by tests/test_gpu_adam.py;
the leaf-direct step is defined as flatten -> flat step -> unflatten."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

H = (7, 1e-3, 0.9, 0.999, 1e-8, 0.0)


@pytest.mark.parametrize("seed", range(4))
def test_leaf_direct_equals_flat_on_random_tables(seed):
    import paper_2211_06934_amd as P
    rng = np.random.default_rng(2000 + seed)
    for case in range(30):
        S = int(rng.integers(1, 100))
        sizes = rng.integers(0, 500, S)
        sizes[rng.random(S) < 0.2] = 0
        sizes[rng.random(S) < 0.2] = rng.integers(1, 6, 1)
        for k in np.nonzero(rng.random(S) < 0.15)[0]:
            sizes[k] = int(rng.integers(2000, 30000))
        if sizes.sum() == 0:
            sizes[0] = 5
        n = int(sizes.sum())
        table = P.segtable_create([int(k) for k in sizes])
        packed = bool(rng.random() < 0.5)

        def tree(src=None):
            if not packed:
                leaves = [torch.empty(int(k), device="cuda") for k in sizes]
            else:
                big, leaves, pos = torch.empty(n + 8 * (S + 1), device="cuda"), [], int(rng.integers(0, 4))
                for k in sizes:
                    leaves.append(big[pos:pos + int(k)])
                    pos += int(k) + int(rng.integers(0, 5))
            if src is not None:
                o = 0
                for x in leaves:
                    x.copy_(src[o:o + x.numel()])
                    o += x.numel()
            return leaves

        g = torch.Generator(device="cuda").manual_seed(int(rng.integers(1 << 30)))
        flat = {k: torch.randn(n, device="cuda", generator=g) * s
                for k, s in (("p", 0.1), ("g", 1e-2), ("m", 1e-3), ("v", 1e-4), ("dP", 1), ("dM", 1), ("dV", 1))}
        flat["v"] = flat["v"].abs()
        trees = {k: tree(v) for k, v in flat.items()}
        trees.update({k: tree() for k in ("po", "mo", "vo", "dg", "dm", "dv")})
        A = {k: P.tree.leaf_pointer_tensor(v, "cuda") for k, v in trees.items()}
        mv = bool(rng.random() < 0.7)
        P.adam_fwd_tree(table, A["p"], A["g"], A["m"], A["v"], *H, A["po"], A["mo"], A["vo"])
        P.adam_bwd_tree(table, A["dP"], A["dM"] if mv else None, A["dV"] if mv else None, A["g"], A["m"], A["v"],
                        *H, A["dg"], A["dm"], A["dv"])
        fo = {k: torch.empty(n, device="cuda") for k in ("po", "mo", "vo", "dg", "dm", "dv")}
        P.adam_fwd(flat["p"], flat["g"], flat["m"], flat["v"], *H, fo["po"], fo["mo"], fo["vo"])
        P.adam_bwd(flat["dP"], flat["dM"] if mv else None, flat["dV"] if mv else None, flat["g"], flat["m"],
                   flat["v"], *H, None, fo["dg"], fo["dm"], fo["dv"])
        torch.cuda.synchronize()
        for k in fo:
            got = torch.cat([x.reshape(-1) for x in trees[k]])
            assert torch.equal(got.view(torch.int32), fo[k].view(torch.int32)), (k, seed, case, S, packed, mv)
        table.close()
