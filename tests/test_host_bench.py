"""CPU checks of bench.py's byte accounting: the interface bytes per element
that the K-step driver must move under each store policy, derived here by
hand from what each launch reads and writes (fp32, 4 bytes per array)."""
import importlib.util
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_whole_trajectory_one_launch():
    b = _bench()
    for K in (1, 3, 5, 16):
        st = b.stored_states(K, "stored")
        # forward: p0, mu0, nu0 and K g in; K (mu, nu) and p_K out
        assert b.fwd_plan(K, st, 16) == (1, 16 + 12 * K)
        # VJP: dP and K (g, mu, nu) in; K dg and dmu0, dnu0 out
        assert b.bwd_plan(K, st, 16) == (1, 12 + 16 * K)


def test_recomputed_trajectory_one_launch():
    b = _bench()
    for K in (1, 3, 8):
        st = b.stored_states(K, "recompute")
        assert st == {K}
        # forward: p0, mu0, nu0, K g in; p_K, mu_K, nu_K out
        assert b.fwd_plan(K, st, 16) == (1, 24 + 4 * K)
        # VJP: dP, mu0, nu0, K g in; K dg, dmu0, dnu0 out
        assert b.bwd_plan(K, st, 16) == (1, 20 + 8 * K)


def test_launch_boundaries():
    b = _bench()
    # K = 10, recompute: state 5 stored as well (two runs of 5 steps).
    # Forward: one launch, two states out.  VJP: run (5, 10] reads state 5
    # (no running dM, dV in), run (0, 5] reads state 0 and the running dM, dV.
    st = b.stored_states(10, "recompute")
    assert st == {5, 10}
    assert b.fwd_plan(10, st, 16) == (1, 16 + 40 + 16)
    assert b.bwd_plan(10, st, 16) == (2, (4 + 8 + 8 + 5 * 8) + (4 + 8 + 8 + 8 + 5 * 8))
    # the same bytes as storing state 8 (runs of 2 and 8)
    assert b.bwd_plan(10, {8, 10}, 16)[1] == b.bwd_plan(10, st, 16)[1]
    assert b.stored_states(17, "recompute") == {5, 11, 17}  # runs of 5, 6, 6
    assert b.stored_states(16, "recompute") == {8, 16}
    # K = 17, whole trajectory: two forward launches (16 + 1 steps), p, mu, nu
    # re-read and p re-written at the boundary; two VJP launches, the second
    # reading the running dM, dV.
    st = b.stored_states(17, "stored")
    assert b.fwd_plan(17, st, 16) == (2, (16 + 16 * 4 + 16 * 8) + (16 + 4 + 8))
    assert b.bwd_plan(17, st, 16) == (2, (4 + 8 + 16 * 16) + (4 + 8 + 8 + 16))
    # the leaf-direct driver launches every 8 steps
    assert b.fwd_plan(9, b.stored_states(9, "stored"), 8)[0] == 2


def test_traffic_record_applies_only_to_its_own_launch_size():
    # a committed counter record is reported only for the kernel sources and
    # the per-launch algorithmic bytes it was taken on (a run with another
    # store policy launches a different amount of work)
    import glob
    import json
    b = _bench()
    recs = sorted(glob.glob(os.path.join(ROOT, "profiles", "traffic_*.json")))
    assert recs
    rec = json.load(open(recs[0]))
    if rec["kernel_src_sha"] != b.kernel_source_sha(rec["kernel"]):
        return  # stale record: reported as null anyway
    alg = rec["algorithmic_bytes_per_launch"]
    assert b.traffic_from_profile(rec["kernel"], rec["workload"], alg) == rec["bytes_per_launch"]
    assert b.traffic_from_profile(rec["kernel"], rec["workload"], alg + 4) is None


def test_documented_paths_exist():
    # every repository path the design notes and the README name must exist
    import re
    for doc in ("DESIGN.md", "README.md"):
        text = open(os.path.join(ROOT, doc)).read()
        for path in sorted(set(re.findall(r"`((?:tests|profiles|oracle|include|paper_2211_06934_amd|workloads)/"
                                          r"[A-Za-z0-9_./{},-]+)`", text))):
            if "{" in path:  # brace lists such as profiles/kernels_{sgd,rmsprop}_treemap.md
                head, alts, tail = re.match(r"(.*)\{([^}]*)\}(.*)", path).groups()
                paths = [head + a + tail for a in alts.split(",")]
            else:
                paths = [path]
            for p in paths:
                assert os.path.exists(os.path.join(ROOT, p.rstrip("/"))), "%s names missing %s" % (doc, p)


def test_kernel_source_lists_name_existing_files():
    b = _bench()
    csrc = os.path.join(ROOT, "paper_2211_06934_amd", "csrc")
    for fam, files in b.KERNEL_SOURCES.items():
        for f in files:
            assert os.path.exists(os.path.join(csrc, f)), (fam, f)
