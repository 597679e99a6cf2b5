"""Concurrent use from two streams.  The library keeps no mutable device
state between calls (no scratch, no counters; the segment table is read
only), so two passes enqueued on two streams at once, sharing one table, must
each give exactly what it gives alone."""
import pytest
import torch

from workloads import HYPER, WORKLOADS

pytestmark = pytest.mark.gpu


def _pass(P, table, numel, seed, stream, K=3):
    g = torch.Generator(device="cuda").manual_seed(seed)
    n = sum(numel)
    with torch.cuda.stream(stream):
        leaves = [[torch.randn(k, device="cuda", generator=g) for k in numel] for _ in range(K + 1)]
        ptr = lambda ls: torch.tensor([x.data_ptr() for x in ls], dtype=torch.int64).cuda()  # noqa: E731
        flats = [torch.empty(n, device="cuda") for _ in range(K + 1)]
        P.tree_flatten_batch(table, [ptr(ls) for ls in leaves], flats)
        mt = [torch.zeros(n, device="cuda")] + [None] * (K - 1) + [torch.empty(n, device="cuda")]
        vt = [torch.zeros(n, device="cuda")] + [None] * (K - 1) + [torch.empty(n, device="cuda")]
        pK = torch.empty(n, device="cuda")
        h = (0, HYPER["lr"], HYPER["b1"], HYPER["b2"], HYPER["eps"], 1e-8)
        P.adam_unrolled_fwd(flats[0], flats[1:], mt, vt, pK, *h)
        cot = torch.randn(n, device="cuda", generator=g)
        dg = [torch.empty(n, device="cuda") for _ in range(K)]
        dm0, dv0 = torch.empty(n, device="cuda"), torch.empty(n, device="cuda")
        P.adam_unrolled_bwd(cot, flats[1:], mt, vt, dg, dm0, dv0, *h)
        outs = [[torch.empty(k, device="cuda") for k in numel] for _ in range(K + 1)]
        P.tree_unflatten_batch(table, [pK] + dg, [ptr(ls) for ls in outs])
    return [leaves, outs, mt[K], vt[K], dm0, dv0]


def _flat(res):
    leaves, outs, *rest = res
    return [x for ls in leaves + outs for x in ls] + rest


def test_two_streams_at_once_equal_alone():
    import paper_2211_06934_amd as P
    numel = WORKLOADS["resnet18_k1"]().numels
    table = P.segtable_create(numel)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    alone = [_pass(P, table, numel, seed, s1) for seed in (1, 2)]
    torch.cuda.synchronize()
    both = [_pass(P, table, numel, 1, s1), _pass(P, table, numel, 2, s2)]  # enqueued back to back, run together
    torch.cuda.synchronize()
    for a, b in zip(alone, both):
        for x, y in zip(_flat(a), _flat(b)):
            assert torch.equal(x.view(torch.int32), y.view(torch.int32))
