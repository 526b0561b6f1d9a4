"""Pins of the oracle's rail-only network (cluster flag `rail_only`; R47, Fig. 2).

In a rail-only network the NIC of local rank r of every node joins rail r, and rails do not
meet: an inter-node transfer between different local ranks first crosses a node's fabric to
the receiver's rank (Fig. 2c).  Pinned: the three cases of Fig. 2 -- inside a node (a) and
across nodes at one rank (b) cost what they cost without rails, across nodes at different
ranks (c) costs exactly one more intra-node hop of the same bytes on the forwarding node; a
cluster of one-device nodes (every device at rank 0) is unchanged; no plan gets faster.
"""
import numpy as np

MAXU = np.uint64(2**64 - 1)


def _cluster(workloads, rail, dpn=4, nodes=2):
    c = workloads.cluster_two_type_8()
    for t in c["types"]:
        t["n_nodes"] = nodes
        t["dev_per_node"] = dpn
    c["rail_only"] = rail
    return c


def _plan(n):
    return dict(hdr=np.zeros(n, np.uint32), cut=np.zeros((16, n), np.uint8), cls=np.zeros((4, n), np.uint32),
                types=np.zeros((4, n), np.uint64))


def _set(p, i, cuts, classes):
    p["hdr"][i] = ((len(cuts) - 1) << 4) | ((len(classes) - 1) << 8)
    for s, c in enumerate(cuts):
        p["cut"][s, i] = c
    for g, (reps, nmb, tv) in enumerate(classes):
        p["cls"][g, i] = reps | (nmb << 16)
        p["types"][g, i] = tv


def test_figure2_cases(oracle_mod, workloads):
    """Two-stage classes, one replica each, placed in (class, stage) order on two 4-device
    nodes per type (A = type 0, B = type 1):
      class 0: A[0] -> A[1]   same node               (Fig. 2a)
      class 1: A[2] -> B[0]   nodes differ, ranks 2/0 (Fig. 2c)
      class 2: B[1] -> A[3]   nodes differ, ranks 1/3 (Fig. 2c)
      class 3: A[4] -> B[2]   nodes differ, ranks 0/2 (Fig. 2c)
    A and B nodes have the same fabric rate and latency here, so every forwarding costs what
    class 0's intra-node hop costs."""
    m = workloads.model("gpt2-small")
    p = _plan(1)
    _set(p, 0, (6, 12), ((1, 2, 0x00), (1, 2, 0x10), (1, 2, 0x01), (1, 2, 0x10)))
    plain = oracle_mod.Oracle(m, _cluster(workloads, False)).detail(p, 0)
    rail = oracle_mod.Oracle(m, _cluster(workloads, True)).detail(p, 0)
    assert plain is not None and rail is not None
    hop = [plain["c"][g][0] for g in range(4)]
    hop_r = [rail["c"][g][0] for g in range(4)]
    intra = hop[0]                                # one intra-node hop of the activation on an A node
    assert hop_r[0] == hop[0]                     # (a)
    assert hop_r[1] == hop[1] + intra             # (c): forwarded over the A node's fabric
    assert hop_r[2] == hop[2] + intra             # (c): over the B node's
    assert hop_r[3] == hop[3] + intra             # (c)
    assert rail["time"] >= plain["time"]


def test_same_rank_pairs_do_not_cross(oracle_mod, workloads):
    """Fig. 2b: every pair at the same local rank in two nodes (A[0..1] -> B[0..1])."""
    m = workloads.model("gpt2-small")
    p = _plan(1)
    _set(p, 0, (6, 12), ((2, 8, 0x10),))
    plain = oracle_mod.Oracle(m, _cluster(workloads, False)).detail(p, 0)
    rail = oracle_mod.Oracle(m, _cluster(workloads, True)).detail(p, 0)
    assert rail["c"] == plain["c"] and rail["time"] == plain["time"]


def test_one_device_nodes_are_unchanged(oracle_mod, workloads):
    """With one device per node every device sits at rank 0: no transfer crosses rails."""
    w = workloads.workload(1)
    m = w["model"]
    a, b = _cluster(workloads, False, dpn=1, nodes=8), _cluster(workloads, True, dpn=1, nodes=8)
    p = workloads.random_plans(m, a, 0x4A11, 0, 3000)
    ta, tb = oracle_mod.Oracle(m, a).eval(p), oracle_mod.Oracle(m, b).eval(p)
    assert np.array_equal(ta, tb)
    assert np.count_nonzero(ta != MAXU) > 1000


def test_forwarding_node(oracle_mod, workloads):
    """A sender on one-device nodes (rank 0) forwards nothing itself: the data crosses the
    receiver's node fabric, so the extra cost follows the receiver's fabric rate."""
    m = workloads.model("gpt2-small")
    c = workloads.cluster_two_type_8()
    c["types"][0].update(n_nodes=4, dev_per_node=1, intra_MBps=0)
    c["types"][1].update(n_nodes=1, dev_per_node=4)
    p = _plan(1)
    _set(p, 0, (6, 12), ((1, 4, 0x11), (1, 4, 0x10)))     # class 0: B[0] -> B[1]; class 1: A[0] -> B[2]
    rates = []
    for MBps in (300_000, 100_000):
        c2 = dict(c, types=[dict(t) for t in c["types"]], rail_only=True)
        c2["types"][1]["intra_MBps"] = MBps
        plain = oracle_mod.Oracle(m, dict(c2, rail_only=False)).detail(p, 0)
        rail = oracle_mod.Oracle(m, c2).detail(p, 0)
        rates.append(rail["c"][1][0] - plain["c"][1][0])
        # class 1: A[0] (rank 0 of a one-device node) -> B[2] (rank 2): crosses at B's node
        assert rail["c"][1][0] > plain["c"][1][0]
    assert rates[1] > rates[0]                            # a slower receiver fabric costs more


def test_rails_never_help(oracle_mod, workloads):
    for idx in (2, 3):
        w = workloads.workload(idx)
        c = dict(w["cluster"], rail_only=True)
        p = workloads.plans(w, 0, 5000)
        t0 = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
        t1 = oracle_mod.Oracle(w["model"], c).eval(p)
        valid = t0 != MAXU
        assert np.array_equal(valid, t1 != MAXU)
        assert np.all(t1[valid] >= t0[valid])
        assert np.count_nonzero(t1[valid] > t0[valid]) > 100
