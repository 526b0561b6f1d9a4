"""Pins of the oracle's per-class layout (each replica class with its own TP degree, pipeline
depth and layer split; Sec. 3 "Non-uniform workload partitioning" and "Resharding").

The DP sync runs per layer segment (the layers between consecutive cuts of any class) on the
coarsest TP layout, after the classes with finer shards have gathered it inside their TP
groups.  Pinned: the per-class encoding of a shared layout gives the shared layout's results;
without links a plan is as slow as its slowest class alone; the segment syncs against the
pinned ring closed form; the resharding all-gather against the ring all-gather closed form.
"""
import numpy as np
import pytest

MAXU = np.uint64(2**64 - 1)


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_per_class_encoding_of_a_shared_layout(oracle_mod, workloads, idx):
    w = workloads.with_memory(workloads.workload(idx), {1: [2, 1], 2: [24, 40, 16]}.get(idx))
    n = min(5000, w["n_plans"])
    p = workloads.plans(w, 0, n)
    h = workloads.as_per_class(p)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    assert np.array_equal(o.eval(p), o.eval(h))
    for i in range(0, n, 97):
        a, b = o.stage_mem(p, i), o.stage_mem(h, i)
        assert (a is None and b is None) or np.array_equal(a, b), i


def _free_links(c):
    for t in c["types"]:
        t.update(intra_MBps=0, pcie_MBps=0, nic_MBps=0, intra_alpha_ps=0, pcie_alpha_ps=0, nic_alpha_ps=0)
    c["nic_MBps_dev"] = None
    c["intra_MBps_node"] = None
    return c


def test_without_links_a_plan_is_its_slowest_class(oracle_mod, workloads):
    """With every link free, classes do not interact: the iteration takes as long as the slowest
    class run alone (its own TP, depth, split, devices and micro-batches)."""
    w = workloads.workload(3)
    c = _free_links({**w["cluster"], "types": [dict(t) for t in w["cluster"]["types"]]})
    m = w["model"]
    p = workloads.het_plans(w, 0, 400)
    o = oracle_mod.Oracle(m, c)
    t = o.eval(p)
    checked = 0
    for i in range(400):
        if t[i] == MAXU:
            continue
        G = ((int(p["hdr"][i]) >> 8) & 3) + 1
        worst = 0
        for g in range(G):
            cw = int(p["chdr"][i]) >> (8 * g) & 0xFF
            tpl, pp = cw & 3, (cw >> 2) + 1
            reps, nmb = int(p["cls"][g, i]) & 0xFFFF, int(p["cls"][g, i]) >> 16
            q = dict(hdr=np.array([tpl | ((pp - 1) << 4)], np.uint32),
                     cut=np.ascontiguousarray(p["ccut"][g * 16:(g + 1) * 16, i:i + 1]),
                     cls=np.array([[reps | (nmb << 16)], [0], [0], [0]], np.uint32),
                     types=np.array([[int(p["types"][g, i])], [0], [0], [0]], np.uint64))
            alone = oracle_mod.Oracle(dict(m, global_batch=nmb * m["mbs"][0]), c).eval(q)[0]
            assert alone != MAXU
            worst = max(worst, int(alone))
        assert int(t[i]) == worst, i
        checked += 1
    assert checked > 200


def _plan(n):
    return dict(hdr=np.zeros(n, np.uint32), cls=np.zeros((4, n), np.uint32), types=np.zeros((4, n), np.uint64),
                chdr=np.zeros(n, np.uint32), ccut=np.zeros((64, n), np.uint8))


def _set(p, i, classes, ep=1, zero=0):
    """classes: (tp, cuts, reps, nmb, type nibbles)"""
    p["hdr"][i] = ((ep.bit_length() - 1) << 2) | ((len(classes) - 1) << 8) | (zero << 10)
    ch = 0
    for g, (tp, cuts, reps, nmb, tv) in enumerate(classes):
        ch |= ((tp.bit_length() - 1) | ((len(cuts) - 1) << 2)) << (8 * g)
        for s, v in enumerate(cuts):
            p["ccut"][g * 16 + s, i] = v
        p["cls"][g, i] = reps | (nmb << 16)
        p["types"][g, i] = tv
    p["chdr"][i] = ch


def _two_type_cluster(workloads):
    c = workloads.cluster_two_type_8()
    for t in c["types"]:
        t["n_nodes"] = 2                      # 8 devices of each type, 4 per node
    return c


def test_segment_syncs(oracle_mod, workloads):
    """Two classes at one TP degree with different layer splits: each layer segment syncs on
    its own ring (the pinned ring closed form on the segment's gradient bytes), and a stage
    waits for the longest segment it holds."""
    m = workloads.model("gpt2-small")
    c = _two_type_cluster(workloads)
    o = oracle_mod.Oracle(m, c)
    p = _plan(1)
    # class 0: 2 replicas on A, split (6, 12); class 1: 2 replicas on B, split (4, 12)
    _set(p, 0, [(1, (6, 12), 2, 4, 0x00), (1, (4, 12), 2, 4, 0x11)])
    d = o.detail(p, 0)
    assert d is not None
    L = m["L"]
    embed = o.param_count(with_head=False) - o.rank_params(1, 1, L)
    head = o.param_count(with_head=True) - o.param_count(with_head=False)
    # inter-node ring over 4 replicas: both types' NICs are 25 GB/s, latency 2 x (0 + 1 us) per step
    alpha = 2 * 1_000_000
    def X(a, b):
        params = o.rank_params(1, 1, b - a) + (embed if a == 0 else 0) + (head if b == L else 0)
        return oracle_mod.dp_sync(4, 0, 4 * params, 2 * params, alpha, 25_000)
    assert d["tdp"][0] == [max(X(0, 4), X(4, 6)), X(6, 12)]
    assert d["tdp"][1] == [X(0, 4), max(X(4, 6), X(6, 12))]
    assert d["time"] == max(d["end"][g][s] + d["tdp"][g][s] for g in range(2) for s in range(2))


def test_resharding_all_gather(oracle_mod, workloads):
    """Classes at TP 1 and TP 4 over the same split: the ring runs on the TP-1 layout, after the
    TP-4 class gathers it inside each TP group -- a ring all-gather over 4 members, each
    contributing its own shard (3 steps of one shard on the node fabric)."""
    m = workloads.model("gpt2-small")
    c = _two_type_cluster(workloads)
    o = oracle_mod.Oracle(m, c)
    p = _plan(2)
    _set(p, 0, [(1, (12,), 4, 4, 0x0), (4, (12,), 1, 4, 0x1)])     # 4 replicas of 1 A, 1 replica of 4 B
    _set(p, 1, [(1, (12,), 4, 4, 0x0), (1, (12,), 1, 4, 0x1)])     # the same, both at TP 1
    L = m["L"]
    full = o.param_count(with_head=True)                            # one stage holds everything at TP 1
    embed4 = m["h"] * (-(-m["vocab"] // 128) * 128) // 4 + m["learned_pos"] * m["h"]
    head4 = m["h"] * (-(-m["vocab"] // 128) * 128) // 4 + m["h"]
    shard4 = o.rank_params(4, 1, L) + embed4 + head4                # one TP-4 rank's parameters
    dp = oracle_mod.dp_sync(5, 0, 4 * full, 2 * full, 2 * 1_000_000, 25_000)
    gather = 3 * 2_000_000 + oracle_mod.link_time(3 * 4 * shard4, oracle_mod.beta_q(300_000))
    d0, d1 = o.detail(p, 0), o.detail(p, 1)
    assert d0["tdp"] == [[dp + gather], [dp + gather]]
    assert d1["tdp"] == [[dp], [dp]]


def test_invalid_per_class_plans(oracle_mod, workloads):
    w = workloads.workload(1)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    p = _plan(7)
    ok = [(1, (6, 12), 2, 4, 0x10), (2, (3, 12), 1, 4, 0x10)]
    _set(p, 0, ok)                                                   # valid
    _set(p, 1, ok); p["hdr"][1] |= 1                                 # header TP field must be 0
    _set(p, 2, ok); p["hdr"][2] |= 1 << 4                            # header PP field must be 0
    _set(p, 3, ok); p["chdr"][3] |= 1 << 14                          # reserved bits of class 1
    _set(p, 4, [(1, (6, 12), 2, 4, 0x10), (2, (3, 11), 1, 4, 0x10)])  # class 1 does not end at L
    _set(p, 5, [(1, (6, 12), 2, 4, 0x10), (8, (12,), 1, 4, 0x0)])    # TP 8 does not divide 12 heads
    _set(p, 6, [(1, (6, 12), 2, 4, 0x10), (4, (3, 12), 1, 4, 0x10)]) # 2 x 1 + 1 x 4 type-A devices > 4
    t = o.eval(p)
    assert t[0] != MAXU
    assert all(t[i] == MAXU for i in range(1, 7)), t


def test_tp_groups_stay_in_a_node(oracle_mod, workloads):
    """Blocks of a pool start at a multiple of their class's TP degree (no TP group spans two
    nodes), so three classes of TP 1, 2 and 1 with one replica each need 5 devices of one
    4-device node -- one more than their sum -- and do not fit; the first two do."""
    w = workloads.workload(1)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    p = _plan(2)
    _set(p, 0, [(1, (12,), 1, 3, 0x0), (2, (12,), 1, 3, 0x0), (1, (12,), 1, 2, 0x0)])
    _set(p, 1, [(1, (12,), 1, 3, 0x0), (2, (12,), 1, 3, 0x0), (1, (12,), 1, 2, 0x1)])
    t = o.eval(p)
    assert t[0] == MAXU and t[1] != MAXU
