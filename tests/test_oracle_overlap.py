"""Pins of the oracle's gradient-sync/backward overlap (header bit 13; R38-R40).

Each stage's gradients are synced in buckets (head, each layer, embedding) that start once
their part of the stage's last backward pass is done, one after another on the stage's DP
ring.  Pinned: a time-ordered event queue over the same buckets (independent code, bucket
syncs from the pinned ring closed form), and the two extremes -- a network so slow that the
buckets run back to back from the first one's readiness, and one so fast that only the last
bucket's sync shows after the stage's end.
"""
import heapq

import numpy as np

MAXU = np.uint64(2**64 - 1)
A_INTRA = 2_000_000          # intra-node message latency of the two-type cluster, ps


def _plan(n):
    return dict(hdr=np.zeros(n, np.uint32), cut=np.zeros((16, n), np.uint8), cls=np.zeros((4, n), np.uint32),
                types=np.zeros((4, n), np.uint64))


def _set(p, i, cuts, classes, tp=1, zero=0, overlap=1):
    p["hdr"][i] = (tp.bit_length() - 1) | ((len(cuts) - 1) << 4) | ((len(classes) - 1) << 8) | (zero << 10) | (
        overlap << 13)
    for s, v in enumerate(cuts):
        p["cut"][s, i] = v
    for g, (reps, nmb, tv) in enumerate(classes):
        p["cls"][g, i] = reps | (nmb << 16)
        p["types"][g, i] = tv


def _queue(jobs):
    """Completion of a first-in-first-out link fed by (ready time, duration) jobs, as a
    time-ordered event simulation."""
    events = [(r, 0, i) for i, (r, _) in enumerate(jobs)]
    heapq.heapify(events)
    free_at, nxt, ready, done = 0, 0, set(), 0
    while events:
        t, _, i = heapq.heappop(events)
        if i >= 0:
            ready.add(i)
        while nxt in ready and free_at <= t:
            free_at = t + jobs[nxt][1]
            done = free_at
            heapq.heappush(events, (free_at, 1, -1))
            nxt += 1
    assert nxt == len(jobs)
    return done


def _stage_jobs(oracle_mod, o, m, d, cuts, s, k, p_all, MBps):
    """(ready time, sync duration) of the buckets of stage s in backward order: head on the last
    stage, layers from the top, embedding on the first stage."""
    S, L, b = len(cuts) - 1, m["L"], m["mbs"][0]
    bk = []
    if s == S - 1:
        bk.append((o.head_time(k, 1, b, True), o.param_count(True) - o.param_count(False)))
    for l in range(cuts[s + 1] - 1, cuts[s] - 1, -1):
        bk.append((o.layer_time(k, 1, b, 1, l, True), o.rank_params(1, 1, 1)))
    if s == 0:
        bk.append((o.embed_time(k, b, True), o.param_count(False) - o.rank_params(1, 1, L)))
    t = d["end"][0][s] - sum(x for x, _ in bk)
    jobs = []
    for comp, P in bk:
        t += comp
        jobs.append((t, oracle_mod.dp_sync(p_all, 0, m["grad_bytes"] * P, m["param_bytes"] * P, A_INTRA, MBps)))
    return jobs


def test_overlap_event_queue_and_extremes(oracle_mod, workloads):
    """Two stages (layers 0-5 on four type-A devices, 6-11 on four type-B ones), four replicas:
    each stage's ring stays inside one node (node latency, node fabric)."""
    m = workloads.model("gpt2-small")
    for MBps in (400, 300_000, 2_500_000):
        c = workloads.cluster_two_type_8()
        for t in c["types"]:
            t["intra_MBps"] = MBps
        o = oracle_mod.Oracle(m, c)
        p = _plan(2)
        _set(p, 0, (6, 12), ((4, 8, 0x10),), overlap=1)
        _set(p, 1, (6, 12), ((4, 8, 0x10),), overlap=0)
        t = o.eval(p)
        d = o.detail(p, 0)
        worst = 0
        for s in range(2):
            jobs = _stage_jobs(oracle_mod, o, m, d, [0, 6, 12], s, s, 4, MBps)
            done = _queue(jobs)
            worst = max(worst, done)
            assert d["tdp"][0][s] == done - d["end"][0][s]
            assert done >= d["end"][0][s] + jobs[-1][1]
            if MBps == 400:                  # communication-bound: back to back from the first bucket
                assert done == jobs[0][0] + sum(x for _, x in jobs)
            if MBps == 2_500_000 and s == 1:  # compute-bound: only the last bucket's sync shows
                assert done == d["end"][0][s] + jobs[-1][1]
        assert int(t[0]) == worst, MBps
        # the same plan without overlap: the stage's whole sync after its end
        d1 = o.detail(p, 1)
        assert int(t[1]) == max(d1["end"][0][s] + d1["tdp"][0][s] for s in range(2))


def test_overlap_needs_the_shared_layout(oracle_mod, workloads):
    w = workloads.workload(1)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    p = dict(hdr=np.array([(1 << 13) | (1 << 8)], np.uint32), cls=np.zeros((4, 1), np.uint32),
             types=np.zeros((4, 1), np.uint64), chdr=np.array([0], np.uint32), ccut=np.zeros((64, 1), np.uint8))
    p["cls"][0, 0] = p["cls"][1, 0] = 4 | 4 << 16
    p["types"][1, 0] = 1
    p["ccut"][0, 0] = p["ccut"][16, 0] = 12
    assert o.eval(p)[0] == MAXU
    p["hdr"][0] &= ~np.uint32(1 << 13)
    assert o.eval(p)[0] != MAXU
    q = _plan(1)
    _set(q, 0, (12,), ((4, 8, 0x0),), overlap=1)
    assert o.eval(q)[0] != MAXU
    q["hdr"][0] |= np.uint32(1 << 14)                         # v = 2: no interleaving with overlap
    assert o.eval(q)[0] == MAXU
