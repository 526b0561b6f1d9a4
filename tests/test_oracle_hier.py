"""Pins of the oracle's two-level all-reduce (cluster flag `ccl_hier`; R50).

With the flag, a dense DP all-reduce whose group fills whole nodes with the same number g > 1
of members per node, over N > 1 nodes (shared layout, no ZeRO), may take the two-level
algorithm: reduce-scatter inside each node, a ring all-reduce of each 1/g shard across the
nodes, all-gather inside each node.  Pinned: the algorithm's time is the composition of two
ring all-reduces of the pinned closed form (g members on the node fabric over the whole
gradient, then N members on the inter-node tier over the 1/g shard); a hand-built plan on two
4-device nodes takes the faster of ring and two-level; groups that are not whole nodes, ZeRO
plans and per-class-layout plans are unchanged; no plan gets slower.
"""
import numpy as np

MAXU = np.uint64(2**64 - 1)


def test_composition_of_two_rings(oracle_mod):
    for g, N, B in ((2, 2, 1000), (4, 2, 10**8), (8, 16, 123456789), (4, 3, 7)):
        for a_in, bw_in, a, bw in ((2_000_000, 300_000, 4_000_000, 25_000), (1000, 900_000, 1000, 50_000)):
            want = (oracle_mod.dp_sync(g, 0, B, 0, a_in, bw_in) +
                    oracle_mod.dp_sync(N, 0, -(-B // g), 0, a, bw))
            assert oracle_mod.hier_allreduce(g, N, B, a_in, bw_in, a, bw) == want


def _cluster(workloads, hier):
    c = workloads.cluster_two_type_8()
    for t in c["types"]:
        t["n_nodes"] = 2                       # two 4-device nodes per type
    c["ccl_hier"] = hier
    return c


def _plan(n):
    return dict(hdr=np.zeros(n, np.uint32), cut=np.zeros((16, n), np.uint8), cls=np.zeros((4, n), np.uint32),
                types=np.zeros((4, n), np.uint64))


def test_whole_nodes_take_the_faster(oracle_mod, workloads):
    """Eight single-device replicas of a one-stage plan on both type-A nodes (g = 4, N = 2):
    the stage's sync is the faster of the 8-member ring and the two-level all-reduce; with
    six replicas the group is not whole nodes and the sync stays the ring."""
    m = dict(workloads.model("gpt2-small"), global_batch=8)
    p = _plan(2)
    for i, reps in enumerate((8, 6)):
        p["hdr"][i] = 0
        p["cut"][0, i] = 12
        p["cls"][0, i] = reps | (8 << 16)
    o0, o1 = oracle_mod.Oracle(m, _cluster(workloads, False)), oracle_mod.Oracle(m, _cluster(workloads, True))
    d0, d1 = o0.detail(p, 0), o1.detail(p, 0)
    P = o0.param_count(with_head=True)
    ring = oracle_mod.dp_sync(8, 0, 4 * P, 2 * P, 2 * 1_000_000, 25_000)
    two = oracle_mod.hier_allreduce(4, 2, 4 * P, 2_000_000, 300_000, 2 * 1_000_000, 25_000)
    assert d0["tdp"][0][0] == ring
    assert d1["tdp"][0][0] == min(ring, two)
    assert two < ring                                     # the fast node fabric carries most of the bytes
    assert o1.detail(p, 1)["tdp"] == o0.detail(p, 1)["tdp"]


def test_selection_properties(oracle_mod, workloads):
    for idx in (2, 4, 5):
        w = workloads.workload(idx)
        c1 = dict(w["cluster"], ccl_hier=True)
        p = workloads.plans(w, 0, 6000)
        t0 = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
        t1 = oracle_mod.Oracle(w["model"], c1).eval(p)
        valid = t0 != MAXU
        assert np.array_equal(valid, t1 != MAXU)
        assert np.all(t1[valid] <= t0[valid])
        zero = ((p["hdr"] >> 10) & 1).astype(bool)
        assert np.array_equal(t1[valid & zero], t0[valid & zero])
        h = workloads.het_plans(w, 0, 2000)
        assert np.array_equal(oracle_mod.Oracle(w["model"], c1).eval(h),
                              oracle_mod.Oracle(w["model"], w["cluster"]).eval(h))
    w = workloads.workload(4)
    p = workloads.plans(w, 0, 6000)
    t0 = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    t1 = oracle_mod.Oracle(w["model"], dict(w["cluster"], ccl_hier=True)).eval(p)
    assert np.count_nonzero(t1 < t0) > 500
