"""Pins of the oracle's tree collectives (cluster flag `ccl_tree`; R48).

With the flag, every DP all-reduce takes the faster of the ring and a pipelined binary tree
(reduce up the tree, broadcast down it); ZeRO's reduce-scatter and all-gather stay rings.
Pinned: the tree's latency term against the rounds of a binomial-tree reduce counted by
brute force; the selection never slows a plan, leaves ZeRO plans and two-member groups (where
the ring always wins) alone, and does speed up many-replica plans of small models.  The tree's
bandwidth term (each gradient crossing the busiest link twice) is a reading, parity unpinned
beyond those properties and GPU = oracle.
"""
import numpy as np

MAXU = np.uint64(2**64 - 1)


def _binomial_reduce_rounds(p):
    """Rounds of a binomial-tree reduce over p members: in each round every member still
    holding a partial sum whose partner (index + step) exists receives it."""
    holding = set(range(p))
    rounds, step = 0, 1
    while len(holding) > 1:
        for i in sorted(holding):
            if i % (2 * step) == 0 and i + step in holding:
                holding.discard(i + step)
        step *= 2
        rounds += 1
    return rounds


def test_latency_term_is_binomial_rounds(oracle_mod):
    """With nothing to send, the tree costs one latency per round up and one per round down."""
    for p in range(2, 70):
        assert oracle_mod.tree_allreduce(p, 0, 1000, 25_000) == 2 * 1000 * _binomial_reduce_rounds(p)
    assert oracle_mod.tree_allreduce(1, 10**9, 1000, 25_000) == 0


def test_tree_against_ring(oracle_mod):
    """Small messages over many members favour the tree, large ones the ring; with two
    members the ring always wins (its bandwidth term is half the tree's)."""
    a, bw = 2_000_000, 25_000
    assert oracle_mod.tree_allreduce(64, 1000, a, bw) < oracle_mod.dp_sync(64, 0, 1000, 0, a, bw)
    assert oracle_mod.tree_allreduce(64, 10**10, a, bw) > oracle_mod.dp_sync(64, 0, 10**10, 0, a, bw)
    for B in (0, 1, 999, 10**6, 10**9):
        assert oracle_mod.tree_allreduce(2, B, a, bw) >= oracle_mod.dp_sync(2, 0, B, 0, a, bw)


def _tree(c):
    return dict(c, ccl_tree=True)


def test_selection_properties(oracle_mod, workloads):
    for idx in (2, 4, 5):
        w = workloads.workload(idx)
        p = workloads.plans(w, 0, 6000)
        t0 = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
        t1 = oracle_mod.Oracle(w["model"], _tree(w["cluster"])).eval(p)
        valid = t0 != MAXU
        assert np.array_equal(valid, t1 != MAXU)
        assert np.all(t1[valid] <= t0[valid])
        zero = ((p["hdr"] >> 10) & 1).astype(bool)
        assert np.array_equal(t1[valid & zero], t0[valid & zero])     # ZeRO stays on rings
        G = ((p["hdr"] >> 8) & 3) + 1
        reps = sum(np.where(G > c, p["cls"][c] & 0xFFFF, 0) for c in range(4))
        small = valid & (reps <= 2)
        assert np.array_equal(t1[small], t0[small])                   # two members: the ring wins


def test_many_small_replicas_get_faster(oracle_mod, workloads):
    """A GPT-2-shaped model of width 256 (about 11M parameters) over 64 one-device replicas: its
    gradient is small against 126 ring latencies, so the tree wins and the sync shrinks."""
    m = dict(workloads.model("gpt2-small"), global_batch=64, h=256, heads=4, kv_heads=4, ffn=1024)
    c = workloads.cluster_two_type_8()
    for t in c["types"]:
        t["n_nodes"] = 8
    p = dict(hdr=np.array([0], np.uint32), cut=np.zeros((16, 1), np.uint8), cls=np.zeros((4, 1), np.uint32),
             types=np.zeros((4, 1), np.uint64))
    p["cut"][0, 0] = 12
    p["cls"][0, 0] = 32 | (32 << 16)
    p["cls"][1, 0] = 32 | (32 << 16)
    p["types"][1, 0] = 1
    p["hdr"][0] = 1 << 8
    d0 = oracle_mod.Oracle(m, c).detail(p, 0)
    d1 = oracle_mod.Oracle(m, _tree(c)).detail(p, 0)
    assert d1["tdp"][0][0] < d0["tdp"][0][0]
    assert d1["time"] < d0["time"]
