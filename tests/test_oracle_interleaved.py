"""Pins of the oracle's interleaved 1F1B (header bits 14-15 = v - 1; R41-R43).

Each device holds v model chunks (virtual stage j S + s on device s) and runs them in the
interleaved order of Narayanan et al. 2021 ("Efficient Large-Scale Language Model Training
on GPU Clusters Using Megatron-LM", Sec. 2.2.2).  Pinned: that paper's bubble closed form,
an event-driven replay of the same op lists (independent code), lower bounds every schedule
obeys, the per-virtual-stage costs against a plain plan over the same cuts, the per-device
DP sync against the ring closed form, and the in-flight activation count.
"""
import numpy as np
import pytest

from oracle import brute_sim

MAXU = np.uint64(2**64 - 1)


@pytest.mark.parametrize("S,v,q", [(2, 2, 2), (2, 4, 3), (3, 2, 2), (4, 2, 4), (4, 4, 2), (5, 3, 2), (8, 2, 2)])
def test_bubble_closed_form(oracle_mod, S, v, q):
    """Uniform chunk costs f, b and free hops: the iteration takes (M v + S - 1)(f + b) --
    M v chunk pairs of useful work per device plus a bubble of (S - 1)/v full-stage pairs."""
    M = q * S
    for fc, bc in ((7, 13), (100, 100), (1, 3)):
        f, b = [fc] * (S * v), [bc] * (S * v)
        want = (M * v + S - 1) * (fc + bc)
        assert max(oracle_mod.pipeline_interleaved(S, v, M, f, b, [0] * (S - 1), 0)) == want
        assert max(brute_sim.simulate_interleaved(S, v, M, f, b, [0] * (S - 1), 0)) == want


def test_against_event_replay():
    """Random non-uniform chunk costs and hops (wrap hop included): the oracle's device sweep
    and the event-driven replay of the same op lists give the same end times per device."""
    from oracle import oracle as O
    rng = np.random.default_rng(41)
    n = 0
    for S in range(2, 9):
        for v in range(2, 5):
            if S * v > 16:
                continue
            for q in (2, 3):
                for _ in range(6):
                    M = q * S
                    f = rng.integers(1, 400, S * v).tolist()
                    b = rng.integers(1, 800, S * v).tolist()
                    c = rng.integers(0, 300, S - 1).tolist()
                    cw = int(rng.integers(0, 300))
                    got = O.pipeline_interleaved(S, v, M, f, b, c, cw)
                    want = brute_sim.simulate_interleaved(S, v, M, f, b, c, cw)
                    assert got == want, (S, v, M, f, b, c, cw)
                    n += 1
    assert n > 100


def test_lower_bounds(oracle_mod):
    """Every device runs all its ops one at a time, and the last device's last backward waits
    for one micro-batch's whole forward-backward chain through all virtual stages."""
    rng = np.random.default_rng(7)
    for _ in range(60):
        S = int(rng.integers(2, 6))
        v = int(rng.integers(2, 16 // S + 1))
        v = min(v, 4)
        M = S * int(rng.integers(2, 4))
        f = rng.integers(1, 500, S * v).tolist()
        b = rng.integers(1, 900, S * v).tolist()
        c = rng.integers(0, 200, S - 1).tolist()
        cw = int(rng.integers(0, 200))
        end = oracle_mod.pipeline_interleaved(S, v, M, f, b, c, cw)
        for s in range(S):
            work = M * sum(f[j * S + s] + b[j * S + s] for j in range(v))
            assert end[s] >= work
        hops = sum(c) * v + cw * (v - 1)
        assert end[0] >= sum(f) + sum(b) + 2 * hops


def test_op_lists_cover_every_pass():
    """Each device runs every micro-batch of each of its chunks once forward and once
    backward, and a micro-batch's forward of a chunk precedes its backward."""
    for S, v, M in ((2, 2, 4), (4, 3, 8), (8, 2, 16), (3, 4, 9)):
        for s in range(S):
            ops = brute_sim.interleaved_op_list(S, v, M, s)
            assert len(ops) == 2 * M * v
            seen = {}
            for i, (kind, vs, m) in enumerate(ops):
                assert vs % S == s
                seen.setdefault((kind, vs, m), i)
            assert len(seen) == 2 * M * v
            for j in range(v):
                for m in range(M):
                    assert seen[("F", j * S + s, m)] < seen[("B", j * S + s, m)]


def _plan(n):
    return dict(hdr=np.zeros(n, np.uint32), cut=np.zeros((16, n), np.uint8), cls=np.zeros((4, n), np.uint32),
                types=np.zeros((4, n), np.uint64))


def _set(p, i, cuts, classes, S, v=1, tp=1, zero=0, overlap=0):
    p["hdr"][i] = (tp.bit_length() - 1) | ((S - 1) << 4) | ((len(classes) - 1) << 8) | (zero << 10) | (
        overlap << 13) | ((v - 1) << 14)
    for s, c in enumerate(cuts):
        p["cut"][s, i] = c
    for g, (reps, nmb, tv) in enumerate(classes):
        p["cls"][g, i] = reps | (nmb << 16)
        p["types"][g, i] = tv


def _cluster(workloads, nodes=4):
    c = workloads.cluster_two_type_8()
    for t in c["types"]:
        t["n_nodes"] = nodes                  # 16 devices of each type, 4 per node
    return c


def test_virtual_stage_costs_and_detail(oracle_mod, workloads):
    """Two devices, two chunks each (cuts 3, 6, 9, 12), one replica on a type-A then a type-B
    device: each virtual stage's forward and backward are those of stage vs of a plain
    four-stage plan over the same cuts with the same device types; the end times are the
    interleaved pipeline over them, the wrap hop being the hop from device 1 back to device 0;
    the iteration is the latest device end plus its sync."""
    m = workloads.model("gpt2-small")
    c = _cluster(workloads)
    o = oracle_mod.Oracle(m, c)
    p = _plan(2)
    M = m["global_batch"] // m["mbs"][0]
    _set(p, 0, (3, 6, 9, 12), ((1, M, 0x10),), S=2, v=2)
    _set(p, 1, (3, 6, 9, 12), ((1, M, 0x1010),), S=4)
    d, dp = o.detail(p, 0), o.detail(p, 1)
    assert d is not None and dp is not None
    assert d["S_class"] == [4] and d["M"] == [M]
    assert d["f"][0] == dp["f"][0] and d["b"][0] == dp["b"][0]
    end = oracle_mod.pipeline_interleaved(2, 2, M, d["f"][0], d["b"][0], d["c"][0][:1], d["c"][0][1])
    assert d["end"][0][:2] == end
    assert d["time"] == max(end[s] + d["tdp"][0][s] for s in range(2))
    assert o.eval(p)[0] == d["time"]


def test_device_sync_over_all_chunks(oracle_mod, workloads):
    """Two replicas of a two-device, two-chunk pipeline, each device position on one node:
    device s syncs the parameters of both its chunks (plus the embedding on device 0 and the
    head on device 1) on one ring over the two replicas."""
    m = workloads.model("gpt2-small")
    c = _cluster(workloads)
    o = oracle_mod.Oracle(m, c)
    Mt = m["global_batch"] // m["mbs"][0]
    p = _plan(1)
    _set(p, 0, (2, 5, 9, 12), ((2, Mt, 0x10),), S=2, v=2)
    d = o.detail(p, 0)
    L = m["L"]
    embed = o.param_count(with_head=False) - o.rank_params(1, 1, L)
    head = o.param_count(with_head=True) - o.param_count(with_head=False)
    # device 0 holds layers 0-1 and 5-8, device 1 layers 2-4 and 9-11; each ring spans two
    # replicas on one 4-device node: node fabric and node latency
    MBps = c["types"][0]["intra_MBps"]
    alpha = c["types"][0]["intra_alpha_ps"]
    p0 = o.rank_params(1, 1, 2 + 4) + embed
    p1 = o.rank_params(1, 1, 3 + 3) + head
    x0 = oracle_mod.dp_sync(2, 0, 4 * p0, 2 * p0, alpha, MBps)
    x1 = oracle_mod.dp_sync(2, 0, 4 * p1, 2 * p1, alpha, MBps)
    assert d["tdp"][0][:2] == [x0, x1]


def test_memory_depends_on_layers_per_device_and_largest_chunk(oracle_mod, workloads):
    """A device's bytes depend on the split only through the layers it holds and its
    largest chunk (activations are counted at that chunk), so two splits that agree on both
    give the same bytes, and each is at least the in-flight passes' activations."""
    m = workloads.model("gpt2-small")
    c = _cluster(workloads)
    o = oracle_mod.Oracle(m, c)
    M = m["global_batch"] // m["mbs"][0]
    per_layer = o.layer_act_bytes(1, m["mbs"][0])
    q = _plan(2)
    _set(q, 0, (2, 5, 9, 12), ((1, M, 0x10),), S=2, v=2)      # device 0: 2 + 4 layers, device 1: 3 + 3
    _set(q, 1, (4, 7, 9, 12), ((1, M, 0x10),), S=2, v=2)      # device 0: 4 + 2 layers, device 1: 3 + 3
    a, b = o.stage_mem(q, 0), o.stage_mem(q, 1)
    assert np.array_equal(a, b)
    for s, big in ((0, 4), (1, 3)):
        assert int(a[0][s]) >= big * per_layer * (2 * (1 - s) + 2 + 1)


def test_in_flight_count_by_difference(oracle_mod, workloads):
    """One more layer in a device's largest chunk adds exactly the in-flight count times one
    layer's activations, plus one layer's state: the count is 2 (S - 1 - s) + (v - 1) S + 1."""
    m = workloads.model("gpt2-small")
    c = _cluster(workloads)
    o = oracle_mod.Oracle(m, c)
    M = m["global_batch"] // m["mbs"][0]
    per_layer = o.layer_act_bytes(1, m["mbs"][0])
    S, v = 2, 3
    # device 0 chunks: layers [0,1), [2,3), [4,6) / [0,1), [2,3), [4,7): one more layer in the
    # largest chunk of device 0 and one fewer in device 1's last chunk (which stays not largest)
    p = _plan(2)
    _set(p, 0, (1, 2, 3, 4, 6, 12), ((1, M, 0x10),), S=S, v=v)
    _set(p, 1, (1, 2, 3, 4, 7, 12), ((1, M, 0x10),), S=S, v=v)
    a, b = o.stage_mem(p, 0), o.stage_mem(p, 1)
    state_one = int(b[0][0]) - int(a[0][0]) - (2 * (S - 1) + (v - 1) * S + 1) * per_layer
    # the state difference is one layer's weights, gradients and optimizer bytes
    layer = o.rank_params(1, 1, 1)
    assert state_one == layer * (m["param_bytes"] + m["grad_bytes"] + m.get("opt_bytes", 12))


def test_invalid_interleaved_plans(oracle_mod, workloads):
    m = workloads.model("gpt2-small")
    c = _cluster(workloads)
    o = oracle_mod.Oracle(m, c)
    Mt = m["global_batch"] // m["mbs"][0]
    p = _plan(8)
    _set(p, 0, (3, 6, 9, 12), ((1, Mt, 0x10),), S=2, v=2)                        # valid
    _set(p, 1, (3, 6, 9, 12), ((1, Mt, 0x10),), S=2, v=2, overlap=1)             # no overlap with v > 1
    _set(p, 2, (6, 12), ((1, Mt, 0x0),), S=1, v=2)                               # one device
    _set(p, 3, (3, 6, 9, 11), ((1, Mt, 0x10),), S=2, v=2)                        # last cut is not L
    _set(p, 4, (3, 6, 12), ((1, Mt, 0x10),), S=2, v=2)                           # S v cuts needed
    _set(p, 5, (3, 6, 9, 12), ((Mt // 2 - 1, Mt, 0x10),), S=2, v=2)              # M = 3 not a multiple of S
    _set(p, 6, (3, 6, 9, 12), ((Mt // 2, Mt, 0x10),), S=2, v=2)                  # M = 2 < 2 S
    p["cut"][:, 7] = np.arange(1, 17) if m["L"] >= 16 else 0
    _set(p, 7, (3, 6, 9, 12), ((1, Mt, 0x10),), S=2, v=2)
    p["hdr"][7] |= np.uint32(1 << 16)                                             # reserved bit
    t = o.eval(p)
    assert t[0] != MAXU
    assert all(t[i] == MAXU for i in range(1, 8)), t
    # the per-class layout does not take interleaving
    h = dict(hdr=np.array([(1 << 14)], np.uint32), cls=np.array([[1 | Mt << 16], [0], [0], [0]], np.uint32),
             types=np.array([[0x10], [0], [0], [0]], np.uint64), chdr=np.array([1 << 2], np.uint32),
             ccut=np.zeros((64, 1), np.uint8))
    h["ccut"][0:4, 0] = (3, 6, 9, 12)
    assert o.eval(h)[0] == MAXU


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_generated_interleaved_plans(oracle_mod, workloads, idx):
    """The seeded generator's interleaved plans are mostly valid, span v = 2..4, and each
    valid one's time is its detail's latest device end plus sync."""
    w = workloads.workload(idx)
    p = workloads.interleaved_plans(w, 0, 3000)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    t = o.eval(p)
    assert np.count_nonzero(t != MAXU) > 2500
    v = ((p["hdr"] >> 14) & 3) + 1
    assert set(np.unique(v)) == {2, 3, 4}
    for i in range(0, 3000, 211):
        d = o.detail(p, i)
        if d is None:
            assert t[i] == MAXU
            continue
        S = ((int(p["hdr"][i]) >> 4) & 15) + 1
        assert d["time"] == int(t[i])
        assert d["time"] == max(d["end"][g][s] + d["tdp"][g][s] for g in range(d["G"]) for s in range(S))
