"""CPU-side checks of the C ABI and the host logic (no kernel is launched).

- the built library exports every entry point include/diffopt.h declares;
- argument validation returns the documented codes and messages before any
  device call;
- the Python tree walk and the workload shapes.
"""
import ctypes
import os
import re
import subprocess

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "diffopt.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(diffopt_[a-z_]+)\s*\(", text)))


def _lib():
    from paper_2211_06934_amd import build
    if not os.path.exists(build.LIB):
        pytest.skip("libdiffopt.so not built")
    return ctypes.CDLL(build.LIB)


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("diffopt_tree_flatten", "diffopt_tree_unflatten", "diffopt_adam_fwd", "diffopt_adam_bwd",
              "diffopt_adam_unrolled_fwd", "diffopt_adam_unrolled_bwd", "diffopt_segtable_create",
              "diffopt_segtable_destroy", "diffopt_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_2211_06934_amd import build
    lib = _lib()
    for name in _declared():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", build.LIB], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (diffopt_\w+)", out))
    assert set(_declared()) <= exported
    # nothing else of ours leaks out under the diffopt_ prefix
    assert exported == set(_declared())


def test_library_has_gfx950_code_only():
    # the offload bundle inside our own build names its target ids
    from paper_2211_06934_amd import build
    _lib()
    blob = open(build.LIB, "rb").read()
    targets = set(re.findall(rb"amdgcn-amd-amdhsa-[-\w:+]*", blob))
    assert targets and all(t.endswith(b"gfx950") for t in targets), targets


def test_validation_errors_before_any_device_call():
    import paper_2211_06934_amd as P
    d = P.diffopt
    lib = d._lib
    f = ctypes.c_void_p(16)  # never dereferenced: every call below fails validation first
    assert lib.diffopt_adam_fwd(f, f, f, f, -1, 0, 1e-3, .9, .999, 1e-8, 0., f, f, f, None, None) == -1
    assert "n must be" in d.last_error()
    assert lib.diffopt_adam_fwd(f, f, f, f, 8, 0, 1e-3, 1.0, .999, 1e-8, 0., f, f, f, None, None) == -1
    assert "b1" in d.last_error()
    assert lib.diffopt_adam_fwd(f, f, f, f, 8, 0, 1e-3, .9, -0.1, 1e-8, 0., f, f, f, None, None) == -1
    assert lib.diffopt_adam_fwd(f, f, f, f, 8, -3, 1e-3, .9, .999, 1e-8, 0., f, f, f, None, None) == -1
    assert lib.diffopt_adam_fwd(f, f, f, f, 8, 0, float("nan"), .9, .999, 1e-8, 0., f, f, f, None, None) == -1
    assert lib.diffopt_adam_fwd(f, f, f, f, 8, 0, 1e-3, .9, .999, -1e-8, 0., f, f, f, None, None) == -1
    assert lib.diffopt_adam_fwd(f, f, f, f, 8, 0, 1e-3, .9, .999, 1e-8, -1., f, f, f, None, None) == -1
    assert lib.diffopt_adam_fwd(None, f, f, f, 8, 0, 1e-3, .9, .999, 1e-8, 0., f, f, f, None, None) == -1
    assert "null" in d.last_error()
    assert lib.diffopt_adam_fwd(ctypes.c_void_p(18), f, f, f, 8, 0, 1e-3, .9, .999, 1e-8, 0., f, f, f, None,
                                None) == -1
    assert "aligned" in d.last_error()
    # n == 0 is a valid no-op even with null buffers
    assert lib.diffopt_adam_fwd(None, None, None, None, 0, 0, 1e-3, .9, .999, 1e-8, 0., None, None, None, None,
                                None) == 0
    assert d.last_error() == ""
    # backward: dmu and dnu both or neither
    assert lib.diffopt_adam_bwd(f, f, None, f, f, f, 8, 0, 1e-3, .9, .999, 1e-8, 0., None, f, f, f, None) == -1
    assert "both" in d.last_error()
    # unrolled: K >= 1
    arr = (ctypes.c_void_p * 2)(16, 16)
    assert lib.diffopt_adam_unrolled_fwd(0, 8, f, arr, arr, arr, f, 0, 1e-3, .9, .999, 1e-8, 0., None) == -1
    assert lib.diffopt_adam_unrolled_bwd(1, 8, f, arr, arr, arr, arr, f, f, 0, 1e-3, .9, .999, 1e-8, 0.,
                                         None) == -1
    assert "distinct" in d.last_error()


def test_trajectory_store_policy_validation_on_host():
    # intermediate moment states may be left unstored (NULL); every call below
    # breaks a rule of the store policy and must fail before any device call
    import paper_2211_06934_amd as P
    d = P.diffopt
    lib = d._lib
    span = int(re.search(r"#define DIFFOPT_REMAT_SPAN (\d+)", open(HEADER).read()).group(1))
    assert span == d.REMAT_SPAN
    K = span + 2
    f, f2 = ctypes.c_void_p(16), ctypes.c_void_p(32)
    full = (ctypes.c_void_p * (K + 1))(*([16] * (K + 1)))
    hole = (ctypes.c_void_p * (K + 1))(*([16] + [None] * (K - 1) + [16]))  # nothing stored between 0 and K
    hyper = (0, 1e-3, .9, .999, 1e-8, 0.)
    # backward: K - 1 > span - 1 consecutive unstored states
    assert lib.diffopt_adam_unrolled_bwd(K, 8, f, full, hole, hole, full, f, f2, *hyper, None) == -1
    assert "every %d-th state" % span in d.last_error()
    # mu stored where nu is not
    mixed = (ctypes.c_void_p * (K + 1))(*([16] * 3 + [None] * (K - 3) + [16]))
    assert lib.diffopt_adam_unrolled_fwd(K, 8, f, full, full, mixed, f, *hyper, None) == -1
    assert "both be stored or both be NULL" in d.last_error()
    # the final state is required by the forward, the initial one by both
    nolast = (ctypes.c_void_p * (K + 1))(*([16] * K + [None]))
    assert lib.diffopt_adam_unrolled_fwd(K, 8, f, full, nolast, nolast, f, *hyper, None) == -1
    assert "final state" in d.last_error()
    nofirst = (ctypes.c_void_p * (K + 1))(*([None] + [16] * K))
    assert lib.diffopt_adam_unrolled_bwd(K, 8, f, full, nofirst, nofirst, full, f, f2, *hyper, None) == -1
    assert "initial state" in d.last_error()
    assert lib.diffopt_adam_unrolled_fwd(K, 8, f, full, nofirst, nofirst, f, *hyper, None) == -1


def test_segtable_validation_and_empty_tables_on_host():
    import paper_2211_06934_amd as P
    with pytest.raises(P.DiffoptError) as ei:
        P.segtable_create([3, -1])
    assert ei.value.code == -1
    with pytest.raises(P.DiffoptError):
        P.segtable_create([3, 4], elem_bytes=3)
    with pytest.raises(P.DiffoptError) as ei:
        P.segtable_create([4, 4], offsets=[0, 2])
    assert "overlap" in str(ei.value)
    with pytest.raises(P.DiffoptError):
        P.segtable_create([4], offsets=[-1])
    # tables with nothing to copy need no device memory
    t = P.segtable_create([0, 0])
    assert t.total == 0 and t.nseg == 2
    t.close()
    t = P.segtable_create([])
    assert t.total == 0 and t.nseg == 0
    lib = P.diffopt._lib
    assert lib.diffopt_segtable_total(None) == -1
    assert lib.diffopt_tree_flatten(None, None, None, None) == -1


def test_tree_walk_roundtrip_on_host():
    from paper_2211_06934_amd.tree import tree_build, tree_leaves
    tree = {"z": [torch.zeros(2), (torch.ones(3), None)], "a": torch.arange(4.0),
            "m": {"k2": torch.zeros(1), "k1": torch.ones(1)}}
    leaves, td = tree_leaves(tree)
    # dict keys sorted, lists/tuples in order
    assert [tuple(x.shape) for x in leaves] == [(4,), (1,), (1,), (2,), (3,)]
    assert torch.equal(leaves[1], torch.ones(1))  # m.k1 before m.k2
    back = tree_build(td, leaves)
    assert back["z"][1][1] is None and isinstance(back["z"][1], tuple)
    assert torch.equal(back["a"], tree["a"])
    assert td.num_leaves == 5


def test_module_tree_uses_registration_order():
    from paper_2211_06934_amd.tree import tree_leaves
    net = torch.nn.Sequential(torch.nn.Linear(3, 4), torch.nn.ReLU(), torch.nn.Linear(4, 2))
    leaves, _ = tree_leaves(net)
    assert [tuple(x.shape) for x in leaves] == [(4, 3), (4,), (2, 4), (2,)]


def test_workload_shapes():
    from workloads import WORKLOADS, many_small_sizes
    assert WORKLOADS["tiny_mlp"]().n == 1761 and WORKLOADS["tiny_mlp"]().nseg == 6
    c = WORKLOADS["convnet32"]()
    assert c.nseg == 576 and c.n == 32 * 112261
    r = WORKLOADS["resnet18_k1"]()
    assert r.nseg == 62 and r.n == 11_689_512
    assert max(r.numels) == 2_359_296 and min(r.numels) == 64
    f = WORKLOADS["flat_1b"]()
    assert f.nseg == 1 and f.n == 1_000_000_000
    s = many_small_sizes()
    assert len(s) == 20000 and min(s) >= 1 and max(s) <= 65536
    assert 1.0e8 < sum(s) < 1.4e8


def test_header_is_plain_c_and_cpp():
    # the boundary is a C ABI: the header must compile as strict C99 and as C++
    for cmd in (["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only", "-x", "c", HEADER],
                ["g++", "-std=c++11", "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only", "-x", "c++",
                 HEADER]):
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_tree_walk_edge_structures_on_host():
    # empty containers and None leaves keep their place; rebuilding with other
    # leaves gives the same structure; unsupported nodes are refused
    from paper_2211_06934_amd.tree import tree_build, tree_leaves
    tree = {"e": [], "t": (), "d": {}, "n": None, "x": [[[torch.ones(2)]], ()], "y": (torch.zeros(0),)}
    leaves, td = tree_leaves(tree)
    assert [tuple(x.shape) for x in leaves] == [(2,), (0,)]  # keys sorted: d, e, n, t, x, y
    back = tree_build(td, [torch.full((2,), 5.0), torch.empty(0)])
    assert back["e"] == [] and back["t"] == () and back["d"] == {} and back["n"] is None
    assert torch.equal(back["x"][0][0][0], torch.full((2,), 5.0)) and back["x"][1] == ()
    assert isinstance(back["y"], tuple) and back["y"][0].numel() == 0
    assert td.num_leaves == 2
    with pytest.raises(TypeError):
        tree_leaves({"a": 3.0})
    with pytest.raises(TypeError):
        tree_leaves([torch.ones(1), "s"])


def test_error_messages_are_per_thread():
    # diffopt_last_error() is thread-local: concurrent failing calls on two
    # host threads each read back their own message
    import threading
    import paper_2211_06934_amd as P
    lib = P.diffopt._lib
    f = ctypes.c_void_p(16)  # never dereferenced: both calls fail validation first
    out = {}
    barrier = threading.Barrier(2)

    def worker(tag):
        for _ in range(200):
            if tag == "count":
                rc = lib.diffopt_adam_fwd(f, f, f, f, 4, -1, 1e-3, .9, .999, 1e-8, 0., f, f, f, None, None)
            else:
                rc = lib.diffopt_adam_fwd(f, f, f, f, 4, 0, 1e-3, 1.5, .999, 1e-8, 0., f, f, f, None, None)
            barrier.wait()
            out.setdefault(tag, []).append((rc, P.diffopt.last_error()))
            barrier.wait()

    ts = [threading.Thread(target=worker, args=(t,)) for t in ("count", "b1")]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert all(rc == -1 and "count" in msg for rc, msg in out["count"])
    assert all(rc == -1 and "b1" in msg for rc, msg in out["b1"])


def test_tree_copy_bindings_check_operand_sizes_on_host():
    # the copy kernels read one address per leaf and table.total flat
    # elements of the table's width: a short address array or a small or
    # narrower flat buffer is refused before any device call
    import paper_2211_06934_amd as P
    d = P.diffopt
    t = d.SegTable(None, [3, 5], None, 4, total=8)  # host-only stand-in: no device table is needed
    ok_ptrs = torch.zeros(2, dtype=torch.int64)
    ok_flat = torch.zeros(8, dtype=torch.float32)
    cases = [
        (torch.zeros(1, dtype=torch.int64), ok_flat, "2 int64 leaf addresses"),
        (torch.zeros(2, dtype=torch.int32), ok_flat, "2 int64 leaf addresses"),
        (ok_ptrs, torch.zeros(7, dtype=torch.float32), "needs 8 elements"),
        (ok_ptrs, torch.zeros(8, dtype=torch.float16), "4-byte elements"),
        (ok_ptrs, torch.zeros(8, dtype=torch.float64), "4-byte elements"),
    ]
    for lp, fl, msg in cases:
        for call in (lambda: P.tree_flatten(t, lp, fl), lambda: P.tree_unflatten(t, fl, lp),
                     lambda: P.tree_flatten_batch(t, [ok_ptrs, lp], [ok_flat, fl]),
                     lambda: P.tree_unflatten_batch(t, [ok_flat, fl], [ok_ptrs, lp])):
            with pytest.raises(ValueError, match=msg):
                call()
    # well-sized host tensors get as far as the device check
    with pytest.raises(ValueError, match="device memory"):
        P.tree_flatten(t, ok_ptrs, ok_flat)
    with pytest.raises(ValueError, match="one entry per tree"):
        P.tree_flatten_batch(t, [ok_ptrs], [ok_flat, ok_flat])
