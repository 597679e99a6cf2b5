"""GPU parity of tree flatten / unflatten (pack / unpack) against the oracle.

Bit-exact for every element size (1, 2, 4, 8 bytes), for dense and gapped
layouts, for leaves whose addresses are out of phase with their flat offsets,
for windows of many tiny leaves (the LDS window bound), leaves holding whole
tiles (the single-entry path) with and without empty leaves, special
fp32 bit patterns, the full 20,000-leaf workload, and small tables on both
sides of the limits of the one-element-per-lane copy.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.support import assert_bits_equal
from workloads import many_small, random_bits, random_shapes, special_f32

pytestmark = pytest.mark.gpu

DT = {1: (np.uint8, torch.uint8), 2: (np.float16, torch.float16), 4: (np.float32, torch.float32),
      8: (np.float64, torch.float64)}


def _np_to_dev(a, tdt):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda").view(tdt)


def _ptrs(leaves):
    return torch.tensor([x.data_ptr() for x in leaves], dtype=torch.int64).cuda()


def _make_leaves(host_leaves, tdt, mode, seed):
    """Device copies of host leaves: separate allocations, or views at random
    element offsets inside one big buffer (arbitrary 16-byte phases)."""
    if mode == "separate":
        return [_np_to_dev(x.reshape(-1), tdt) if x.size else torch.empty(0, dtype=tdt, device="cuda")
                for x in host_leaves]
    rng = np.random.default_rng(seed)
    total = sum(x.size for x in host_leaves) + 16 * (len(host_leaves) + 1)
    big = torch.zeros(total, dtype=tdt, device="cuda")
    out = []
    pos = int(rng.integers(0, 8))
    for x in host_leaves:
        view = big[pos:pos + x.size]
        if x.size:
            view.copy_(_np_to_dev(x.reshape(-1), tdt))
        out.append(view)
        pos += x.size + int(rng.integers(0, 9))
    return out


def _roundtrip(host_leaves, eb, mode, seed, offsets=None):
    import paper_2211_06934_amd as P
    ndt, tdt = DT[eb]
    numel = [x.size for x in host_leaves]
    table = P.segtable_create(numel, offsets, eb)
    n = table.total
    leaves = _make_leaves(host_leaves, tdt, mode, seed)
    fill = random_bits(max(n, 1), ndt, seed + 7)[:n]
    flat = _np_to_dev(fill, tdt)  # gaps must keep these bits
    P.tree_flatten(table, _ptrs(leaves), flat)
    torch.cuda.synchronize()
    expect = np.array(fill, copy=True)
    ref = oracle.pack([x.reshape(-1) for x in host_leaves], flat_len=n, offsets=offsets, dtype=ndt)
    if offsets is None:
        expect = ref
    else:
        for o, x in zip(offsets, host_leaves):
            expect[o:o + x.size] = x.reshape(-1)
        covered = np.zeros(n, bool)
        for o, x in zip(offsets, host_leaves):
            covered[o:o + x.size] = True
        assert_bits_equal(ref[covered], expect[covered], "oracle")
    got = flat.cpu().numpy().view(ndt)
    assert_bits_equal(got, expect, "flatten")

    # unflatten into fresh leaves of the same layout mode, compare with the oracle
    outs = _make_leaves([np.zeros_like(x) for x in host_leaves], tdt, mode, seed + 1)
    P.tree_unflatten(table, flat, _ptrs(outs))
    torch.cuda.synchronize()
    ref_leaves = oracle.unpack(expect, [x.shape for x in host_leaves], offsets=offsets)
    for i, (o, r) in enumerate(zip(outs, ref_leaves)):
        assert_bits_equal(o.cpu().numpy().view(ndt).reshape(-1), r.reshape(-1), "unflatten leaf %d" % i)
    table.close()


@pytest.mark.parametrize("eb", [4, 1, 2, 8])
@pytest.mark.parametrize("mode", ["separate", "packed-views"])
def test_random_trees_bit_exact(eb, mode):
    shapes = random_shapes(400, 3000, seed=eb)
    ndt = DT[eb][0]
    leaves = [random_bits(int(np.prod(s)), ndt, seed=100 * eb + i).reshape(s) for i, s in enumerate(shapes)]
    _roundtrip(leaves, eb, mode, seed=eb)


@pytest.mark.parametrize("eb", [4, 2])
def test_explicit_offsets_with_gaps(eb):
    rng = np.random.default_rng(3)
    ndt = DT[eb][0]
    leaves = [random_bits(int(k), ndt, seed=int(k) + i) for i, k in
              enumerate(rng.integers(0, 3000, size=120))]
    order = rng.permutation(len(leaves))  # table order differs from flat order
    offsets = [0] * len(leaves)
    pos = int(rng.integers(0, 5))
    for j in order:
        offsets[j] = pos
        pos += leaves[j].size + int(rng.integers(0, 7))
    _roundtrip(leaves, eb, "packed-views", seed=11, offsets=offsets)


@pytest.mark.parametrize("eb", [4, 1, 2, 8])
@pytest.mark.parametrize("mode", ["separate", "packed-views"])
@pytest.mark.parametrize("with_empty", [False, True])
@pytest.mark.parametrize("layout", ["dense", "permuted-gaps"])
def test_large_leaves_bit_exact(eb, mode, with_empty, layout):
    # Leaves of 40 KiB and more hold whole tiles (8 KiB of destination each),
    # which the kernel copies from a single table entry read into scalar
    # registers; the tiny leaves between them give tiles that span several
    # leaves. Empty leaves make the table index differ from the leaf index;
    # explicit offsets in another order than the table's, with gaps, put the
    # leaves at arbitrary phases of the flat buffer's lines.
    rng = np.random.default_rng(20 + eb)
    ndt = DT[eb][0]
    sizes = []
    for k in range(9):
        sizes.append((40 << 10) // eb + int(rng.integers(0, 3000)))
        sizes.append(int(rng.integers(1, 40)))
        if with_empty:
            sizes.append(0)
    leaves = [random_bits(k, ndt, seed=300 + 7 * eb + i) for i, k in enumerate(sizes)]
    offsets = None
    if layout == "permuted-gaps":
        order = rng.permutation(len(leaves))
        offsets = [0] * len(leaves)
        pos = int(rng.integers(0, 5))
        for j in order:
            offsets[j] = pos
            pos += leaves[j].size + int(rng.integers(0, 7))
    _roundtrip(leaves, eb, mode, seed=40 + eb, offsets=offsets)


SMALL_TABLES = {  # at most 32 nonempty leaves and 2^16 elements, no gaps: one element per lane
    "one-leaf": [1761],
    "ragged-with-empties": [0, 3, 40, 1, 1600, 0, 40, 7, 1, 4096, 5, 2, 0],
    "32-leaves": [(7 * k) % 23 + 1 for k in range(32)],
    "33-leaves (tiled)": [(7 * k) % 23 + 1 for k in range(33)],
    "2^16-elements": [1 << 15, 1, (1 << 15) - 4, 3],
    "2^16+1-elements (tiled)": [1 << 15, 2, (1 << 15) - 4, 3],
    "sparse-40-leaves": [0 if k % 4 else 3 * k + 1 for k in range(40)],  # 10 nonempty, indices up to 36
}


@pytest.mark.parametrize("eb", [4, 1, 2, 8])
@pytest.mark.parametrize("mode", ["separate", "packed-views"])
@pytest.mark.parametrize("case", list(SMALL_TABLES))
def test_small_tables_bit_exact(case, mode, eb):
    ndt = DT[eb][0]
    leaves = [random_bits(k, ndt, seed=31 * eb + i) for i, k in enumerate(SMALL_TABLES[case])]
    _roundtrip(leaves, eb, mode, seed=eb + 5)


@pytest.mark.parametrize("gap", [0, 3])
def test_small_table_with_explicit_offsets(gap):
    # offsets equal to the concatenation keep the one-element-per-lane copy;
    # a gap makes the layout other than the concatenation (the tiled kernel)
    numel = [40, 0, 1600, 7, 1]
    leaves = [random_bits(k, np.float32, seed=70 + i) for i, k in enumerate(numel)]
    offsets, pos = [], 0
    for k in numel:
        offsets.append(pos)
        pos += k + (gap if k else 0)
    _roundtrip(leaves, 4, "separate", seed=9, offsets=offsets)


def test_special_values_survive():
    sp = special_f32()
    leaves = [np.tile(sp, k)[: (k * 5) % 41 + 1] for k in range(1, 60)]
    _roundtrip(leaves, 4, "packed-views", seed=5)
    _roundtrip(leaves, 4, "separate", seed=6)


@pytest.mark.parametrize("size", [1, 2, 3, 5])
def test_window_of_tiny_leaves(size):
    # 20,000 tiny leaves: every tile holds the largest window of leaves the
    # LDS staging allows, plus empty leaves sprinkled between them.
    shapes = []
    for i in range(20000):
        shapes.append((0,) if i % 13 == 0 else (size + (i % 3 == 0),))
    leaves = [random_bits(int(np.prod(s)), np.float32, seed=i % 1000).reshape(s) for i, s in enumerate(shapes)]
    _roundtrip(leaves, 4, "separate" if size % 2 else "packed-views", seed=size)


def test_edge_tables():
    import paper_2211_06934_amd as P
    # no leaves, all-empty leaves: no-ops with total 0
    for numel in ([], [0, 0, 0]):
        t = P.segtable_create(numel)
        assert t.total == 0 and t.nseg == len(numel)
        f = torch.empty(0, dtype=torch.float32, device="cuda")
        P.tree_flatten(t, torch.zeros(len(numel), dtype=torch.int64, device="cuda"), f)
        P.tree_unflatten(t, f, torch.zeros(len(numel), dtype=torch.int64, device="cuda"))
    # a single leaf is a plain copy, odd length, both layouts
    x = random_bits(1_000_003, np.float32, seed=1)
    _roundtrip([x], 4, "separate", seed=1)
    _roundtrip([x], 4, "packed-views", seed=2)
    # overlap is rejected
    with pytest.raises(P.DiffoptError):
        P.segtable_create([4, 4], [0, 3])
    torch.cuda.synchronize()


def test_python_tree_api_roundtrip():
    import paper_2211_06934_amd as P
    torch.manual_seed(0)
    tree = {"b": [torch.randn(3, 5, device="cuda"), torch.randn(7, device="cuda")],
            "a": (torch.randn(1, device="cuda"), {"z": torch.randn(2, 2, 2, device="cuda"), "y": None}),
            "c": torch.randn(0, device="cuda")}
    flat, spec = P.tree.flatten(tree)
    leaves, _ = P.tree.tree_leaves(tree)
    assert torch.equal(flat, torch.cat([x.reshape(-1) for x in leaves]))
    back = P.tree.unflatten(flat, spec)
    assert torch.equal(back["b"][0], tree["b"][0]) and torch.equal(back["a"][1]["z"], tree["a"][1]["z"])
    assert back["a"][1]["y"] is None and isinstance(back["a"], tuple)


@pytest.mark.parametrize("raw", [False, True])
def test_python_tree_api_on_a_side_stream(raw):
    # the copies run on the given stream (a torch stream or a raw hipStream_t
    # address); the leaf-address arrays are allocated on that stream too
    import paper_2211_06934_amd as P
    torch.manual_seed(1)
    tree = [torch.randn(k, device="cuda") for k in (5, 4096 + 3, 1, 70000)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    s = side.cuda_stream if raw else side
    flat = torch.empty(sum(x.numel() for x in tree), device="cuda")
    flat, spec = P.tree.flatten(tree, out=flat, stream=s)
    outs = [torch.empty_like(x) for x in tree]
    back = P.tree.unflatten(flat, spec, out_leaves=outs, stream=s)
    side.synchronize()
    assert torch.equal(flat, torch.cat(tree))
    assert all(torch.equal(a, b) for a, b in zip(back, tree))


def test_many_small_full_size_bit_exact():
    # The 20,000-leaf workload at full size: flatten separately allocated leaves,
    # compare the whole flat buffer with the oracle's pack, then unflatten.
    import paper_2211_06934_amd as P
    w = many_small()
    numel = w.numels
    n = w.n
    src = torch.empty(n, dtype=torch.float32, device="cuda")
    src.view(torch.int32).random_(generator=torch.Generator(device="cuda").manual_seed(9))
    leaves = list(torch.split(src.clone(), numel))
    leaves = [x.clone() for x in leaves]  # separate allocations
    table = P.segtable_create(numel)
    assert table.total == n
    flat = torch.empty(n, dtype=torch.float32, device="cuda")
    P.tree_flatten(table, _ptrs(leaves), flat)
    torch.cuda.synchronize()
    host_leaves = [x.cpu().numpy() for x in leaves]
    ref = oracle.pack(host_leaves)
    assert_bits_equal(flat.cpu().numpy(), ref, "flatten 20k")
    outs = [torch.empty_like(x) for x in leaves]
    P.tree_unflatten(table, flat, _ptrs(outs))
    torch.cuda.synchronize()
    got = torch.cat(outs).cpu().numpy()
    assert_bits_equal(got, np.concatenate(host_leaves), "unflatten 20k")


@pytest.mark.parametrize("eb", [4, 1, 8])
@pytest.mark.parametrize("ntrees", [1, 3, 16, 17, 40])
def test_batched_copies_bit_exact(eb, ntrees):
    # ntrees trees of one structure in one call (one launch per 16 trees):
    # every tree's flat buffer equals the oracle's pack of its leaves, and
    # the batched unflatten rebuilds every tree, bit for bit; gaps between
    # leaves (explicit offsets) keep the flat buffer's bits
    import paper_2211_06934_amd as P
    ndt, tdt = DT[eb]
    rng = np.random.default_rng(eb * 100 + ntrees)
    numel = [0, 3] + [int(k) for k in rng.integers(0, 2500, size=60)] + [0, 4096 + 1]
    offsets, pos = [], 0
    for k in numel:
        pos += int(rng.integers(0, 5))
        offsets.append(pos)
        pos += k
    table = P.segtable_create(numel, offsets, eb)
    n = table.total
    host = [[random_bits(k, ndt, seed=1000 * t + j) for j, k in enumerate(numel)] for t in range(ntrees)]
    trees = [_make_leaves(h, tdt, "packed-views" if t % 2 else "separate", seed=t) for t, h in enumerate(host)]
    fills = [random_bits(max(n, 1), ndt, seed=77 + t)[:n] for t in range(ntrees)]
    flats = [_np_to_dev(f, tdt) for f in fills]
    P.tree_flatten_batch(table, [_ptrs(x) for x in trees], flats)
    outs = [_make_leaves([np.zeros(k, ndt) for k in numel], tdt, "separate", seed=50 + t) for t in range(ntrees)]
    P.tree_unflatten_batch(table, flats, [_ptrs(x) for x in outs])
    torch.cuda.synchronize()
    for t in range(ntrees):
        expect = np.array(fills[t], copy=True)
        packed = oracle.pack(host[t], flat_len=n, offsets=offsets, dtype=ndt)
        for o, k in zip(offsets, numel):
            expect[o:o + k] = packed[o:o + k]
        assert_bits_equal(flats[t].cpu().numpy().view(ndt), expect, "flatten tree %d" % t)
        for j, (o, r) in enumerate(zip(outs[t], host[t])):
            assert_bits_equal(o.cpu().numpy().view(ndt), r, "unflatten tree %d leaf %d" % (t, j))
    # no trees is a no-op; mismatched lists are refused before any launch
    P.tree_flatten_batch(table, [], [])
    with pytest.raises(ValueError):
        P.tree_unflatten_batch(table, flats[:1], [])
    table.close()


def test_binding_enqueues_on_the_current_stream():
    # the binding reads torch's current stream through the raw accessor; it
    # must be the stream torch itself reports, also inside a stream context
    import paper_2211_06934_amd as P
    d = P.diffopt
    assert d._stream(None) == torch.cuda.current_stream().cuda_stream
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        assert d._stream(None) == side.cuda_stream == torch.cuda.current_stream().cuda_stream
    assert d._stream(None) == torch.cuda.current_stream().cuda_stream


@pytest.mark.parametrize("dtype", [torch.float16, torch.bfloat16, torch.float64, torch.int8, torch.int64])
def test_python_tree_api_other_dtypes(dtype):
    # the table follows the leaves' element size (1, 2, 4 or 8 bytes); the
    # copies move bits, so every dtype round-trips exactly
    import paper_2211_06934_amd as P
    g = torch.Generator(device="cuda").manual_seed(3)
    shapes = [(3, 5), (7,), (0,), (1,), (33, 3)]
    if dtype.is_floating_point:
        leaves = [torch.randn(s, device="cuda", generator=g).to(dtype) for s in shapes]
    else:
        leaves = [torch.randint(-100, 100, s, device="cuda", generator=g).to(dtype) for s in shapes]
    tree = {"w": leaves[:2], "e": leaves[2], "b": tuple(leaves[3:])}
    flat, spec = P.tree.flatten(tree)
    order, _ = P.tree.tree_leaves(tree)
    assert flat.dtype == dtype and flat.numel() == sum(x.numel() for x in leaves)
    assert torch.equal(flat, torch.cat([x.reshape(-1) for x in order]))
    back = P.tree.unflatten(flat, spec)
    for a, b in zip(P.tree.tree_leaves(back)[0], order):
        assert a.dtype == dtype and a.shape == b.shape and torch.equal(a, b)
