"""Randomized bit-exact parity of tree flatten / unflatten against the oracle.

Three hundred seeded random tables: every element size, empty, tiny and large
leaves (large ones hold whole tiles, copied from one table entry; the rest
give windows of several leaves), dense offsets or explicit offsets in a
permuted order with gaps, leaves as separate allocations or as views at
random phases inside one buffer.  Flatten must reproduce the oracle's pack
(and leave the gaps' bits alone); unflatten must return every leaf bit for
bit.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.support import assert_bits_equal
from workloads import random_bits

pytestmark = pytest.mark.gpu

DT = {1: (np.uint8, torch.uint8), 2: (np.float16, torch.float16), 4: (np.float32, torch.float32),
      8: (np.float64, torch.float64)}


def _dev(a, tdt):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda").view(tdt)


def _leaves(arrs, tdt, packed, rng):
    if not packed:
        return [_dev(a, tdt) if a.size else torch.empty(0, dtype=tdt, device="cuda") for a in arrs]
    big = torch.zeros(sum(a.size for a in arrs) + 16 * (len(arrs) + 1), dtype=tdt, device="cuda")
    out, pos = [], int(rng.integers(0, 8))
    for a in arrs:
        v = big[pos:pos + a.size]
        if a.size:
            v.copy_(_dev(a, tdt))
        out.append(v)
        pos += a.size + int(rng.integers(0, 9))
    return out


def _ptrs(leaves):
    return torch.tensor([x.data_ptr() for x in leaves], dtype=torch.int64).cuda()


@pytest.mark.parametrize("seed", range(6))
def test_random_tables_bit_exact(seed):
    import paper_2211_06934_amd as P
    rng = np.random.default_rng(1000 + seed)
    for case in range(50):
        eb = int(rng.choice([1, 2, 4, 8]))
        ndt, tdt = DT[eb]
        S = int(rng.integers(1, 120))
        sizes = rng.integers(0, 600, S)
        sizes[rng.random(S) < 0.25] = 0
        sizes[rng.random(S) < 0.2] = rng.integers(1, 5, 1)
        for k in np.nonzero(rng.random(S) < 0.15)[0]:
            sizes[k] = int(rng.integers(2000, 60000)) // eb
        offsets = None
        if rng.random() < 0.4:
            offsets, pos = [0] * S, int(rng.integers(0, 9))
            for j in rng.permutation(S):
                offsets[j] = pos
                pos += int(sizes[j]) + int(rng.integers(0, 9))
        table = P.segtable_create([int(k) for k in sizes], offsets, eb)
        n = table.total
        host = [random_bits(int(k), ndt, seed=int(rng.integers(1 << 30))) for k in sizes]
        packed = bool(rng.random() < 0.5)
        leaves = _leaves(host, tdt, packed, rng)
        fill = random_bits(max(n, 1), ndt, seed=5 + case)[:n]
        flat = _dev(fill, tdt)  # gaps must keep these bits
        P.tree_flatten(table, _ptrs(leaves), flat)
        torch.cuda.synchronize()
        ref = oracle.pack(host, flat_len=n, offsets=offsets, dtype=ndt)
        offs = offsets if offsets is not None else [int(x) for x in np.concatenate([[0], np.cumsum(sizes)[:-1]])]
        expect = np.array(fill, copy=True)
        for o, a in zip(offs, host):
            expect[o:o + a.size] = ref[o:o + a.size]
        assert_bits_equal(flat.cpu().numpy().view(ndt), expect, "flatten, seed %d case %d" % (seed, case))
        outs = _leaves([np.zeros_like(a) for a in host], tdt, packed, rng)
        P.tree_unflatten(table, flat, _ptrs(outs))
        torch.cuda.synchronize()
        back = oracle.unpack(expect, [a.shape for a in host], offsets=offsets)
        for i, (o, r) in enumerate(zip(outs, back)):
            assert_bits_equal(o.cpu().numpy().view(ndt).reshape(-1), r.reshape(-1),
                              "unflatten leaf %d, seed %d case %d" % (i, seed, case))
        table.close()
