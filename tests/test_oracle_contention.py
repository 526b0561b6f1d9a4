"""Pins of the oracle's link contention (cluster flag `contention`; R49).

With the per-class layout a stage can hold several layer segments, whose syncs run at the
same time over the same devices (R37).  With contention their link times add up while their
latencies overlap: the stage waits for the largest latency part plus the sum of the link-time
parts.  Pinned: the two parts against the ring closed form (2 (p - 1) latencies, 2 (p - 1)
chunks of ceil(B / p) bytes on the slowest link) on a hand-built two-class plan; plans whose
stages hold one segment each (every shared-layout plan) are unchanged, also with the tree and
two-level all-reduce enabled; no plan gets faster.
"""
import numpy as np

MAXU = np.uint64(2**64 - 1)


def _plan(n):
    return dict(hdr=np.zeros(n, np.uint32), cls=np.zeros((4, n), np.uint32), types=np.zeros((4, n), np.uint64),
                chdr=np.zeros(n, np.uint32), ccut=np.zeros((64, n), np.uint8))


def _set(p, i, classes):
    """classes: (tp, cuts, reps, nmb, type nibbles)"""
    p["hdr"][i] = (len(classes) - 1) << 8
    ch = 0
    for g, (tp, cuts, reps, nmb, tv) in enumerate(classes):
        ch |= ((tp.bit_length() - 1) | ((len(cuts) - 1) << 2)) << (8 * g)
        for s, v in enumerate(cuts):
            p["ccut"][g * 16 + s, i] = v
        p["cls"][g, i] = reps | (nmb << 16)
        p["types"][g, i] = tv
    p["chdr"][i] = ch


def test_segments_of_a_stage_share_its_links(oracle_mod, workloads):
    """Class 0 splits at (6, 12), class 1 at (4, 12): segments [0, 4), [4, 6), [6, 12). Stage
    0 of class 0 holds the first two, stage 1 of class 1 the last two; each ring spans the 4
    replicas across nodes (inter-node latency 2 x 1 us, 25 GB/s NICs)."""
    m = workloads.model("gpt2-small")
    c = workloads.cluster_two_type_8()
    for t in c["types"]:
        t["n_nodes"] = 2
    p = _plan(1)
    _set(p, 0, [(1, (6, 12), 2, 4, 0x00), (1, (4, 12), 2, 4, 0x11)])
    d0 = oracle_mod.Oracle(m, c).detail(p, 0)
    d1 = oracle_mod.Oracle(m, dict(c, contention=True)).detail(p, 0)
    L = m["L"]
    o = oracle_mod.Oracle(m, c)
    embed = o.param_count(with_head=False) - o.rank_params(1, 1, L)
    head = o.param_count(with_head=True) - o.param_count(with_head=False)
    alpha, bq = 2 * 1_000_000, oracle_mod.beta_q(25_000)

    def parts(a, b):
        params = o.rank_params(1, 1, b - a) + (embed if a == 0 else 0) + (head if b == L else 0)
        lat = 2 * 3 * alpha
        bw = oracle_mod.link_time(2 * 3 * (-(-4 * params // 4)), bq)
        assert lat + bw == oracle_mod.dp_sync(4, 0, 4 * params, 2 * params, alpha, 25_000)
        return lat, bw
    (la, ba), (lb, bb), (lc, bc) = parts(0, 4), parts(4, 6), parts(6, 12)
    assert d0["tdp"][0] == [max(la + ba, lb + bb), lc + bc]
    assert d1["tdp"][0] == [max(la, lb) + ba + bb, lc + bc]
    assert d1["tdp"][1] == [la + ba, max(lb, lc) + bb + bc]
    assert d1["time"] >= d0["time"]


def test_one_segment_per_stage_is_unchanged(oracle_mod, workloads):
    for idx in (2, 4, 5):
        w = workloads.workload(idx)
        p = workloads.plans(w, 0, 4000)
        a = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
        b = oracle_mod.Oracle(w["model"], dict(w["cluster"], contention=True)).eval(p)
        assert np.array_equal(a, b)
        h = workloads.as_per_class(p)
        assert np.array_equal(oracle_mod.Oracle(w["model"], dict(w["cluster"], contention=True)).eval(h), a)


def test_one_segment_per_stage_with_other_algorithms(oracle_mod, workloads):
    """With the tree and two-level all-reduce also enabled, a stage that holds one segment keeps
    the sync the faster algorithm gives: contention changes no shared-layout plan of any kind
    (plain, overlapped, zero-bubble, interleaved)."""
    for idx in (2, 3, 4, 5):
        w = workloads.workload(idx)
        c = dict(w["cluster"], ccl_tree=True, ccl_hier=True, rail_only=True)
        p = workloads.plans(w, 0, 3000)
        p["hdr"][1000:2000] |= np.uint32(1 << 13)
        p["hdr"][2000:] |= np.uint32(1 << 16)
        q = workloads.interleaved_plans(w, 0, 1000)
        for x in (p, q):
            a = oracle_mod.Oracle(w["model"], c).eval(x)
            b = oracle_mod.Oracle(w["model"], dict(c, contention=True)).eval(x)
            assert np.array_equal(a, b), idx
        assert np.any(a != oracle_mod.Oracle(w["model"], w["cluster"]).eval(q))


def test_contention_never_helps(oracle_mod, workloads):
    for idx in (2, 3, 4):
        w = workloads.workload(idx)
        p = workloads.het_plans(w, 0, 4000)
        a = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
        b = oracle_mod.Oracle(w["model"], dict(w["cluster"], contention=True)).eval(p)
        valid = a != MAXU
        assert np.array_equal(valid, b != MAXU)
        assert np.all(b[valid] >= a[valid])
        assert np.count_nonzero(b[valid] > a[valid]) > 100
