"""Pins of the oracle's zero-bubble order (header bit 16; R44-R46).

The backward pass splits into B (input gradient, what the previous stage waits for) and W
(weight gradient, local); stage s runs the 1F1B order of forwards and B passes and releases
each W s micro-batches after its B (ZB-H1 of Qi et al. 2024, "Zero Bubble Pipeline
Parallelism"), W being half of the stage's backward compute (the MoE all-to-all stays in B).  Pinned: that paper's ZB-H1 bubble
(S - 1)(F + B - W) for equal pass costs, an
event-driven replay of the same op lists (independent code), the reduction to 1F1B when W
costs nothing, the in-flight count (every stage at most S micro-batches, 1F1B's peak) against a
walk of the op lists, the per-stage split of the backward, and the invalid combinations.
"""
import numpy as np
import pytest

from oracle import brute_sim

MAXU = np.uint64(2**64 - 1)


@pytest.mark.parametrize("S", [2, 3, 4, 6, 8])
def test_bubble_closed_form(oracle_mod, S):
    """Equal forward, input-gradient and weight-gradient costs (and free hops): the iteration
    takes M (F + B + W) + (S - 1)(F + B - W), against 1F1B's M (F + B') + (S - 1)(F + B') with
    B' = B + W."""
    for M in (S, 2 * S, 3 * S + 1):
        for x in (1, 7, 100):
            f = b = w = [x] * S
            got = max(oracle_mod.pipeline_zb(S, M, f, b, w, [0] * (S - 1)))
            assert got == M * 3 * x + (S - 1) * x
            plain = max(oracle_mod.pipeline(S, M, f, [2 * x] * S, [0] * (S - 1)))
            assert plain == M * 3 * x + (S - 1) * 3 * x


def test_against_event_replay():
    from oracle import oracle as O
    rng = np.random.default_rng(44)
    for _ in range(400):
        S = int(rng.integers(1, 9))
        M = int(rng.integers(1, 3 * S + 3))
        f = rng.integers(1, 500, S).tolist()
        b = rng.integers(1, 500, S).tolist()
        w = rng.integers(0, 500, S).tolist()
        c = rng.integers(0, 300, S).tolist()
        assert O.pipeline_zb(S, M, f, b, w, c[:S - 1]) == brute_sim.simulate_zb(S, M, f, b, w, c), (S, M)


def test_free_weight_gradient_is_1f1b(oracle_mod):
    """With W = 0 the order is 1F1B's with B as the backward pass."""
    rng = np.random.default_rng(45)
    for _ in range(200):
        S = int(rng.integers(1, 9))
        M = int(rng.integers(1, 3 * S + 3))
        f = rng.integers(1, 500, S).tolist()
        b = rng.integers(1, 500, S).tolist()
        c = rng.integers(0, 300, max(S - 1, 0)).tolist()
        assert oracle_mod.pipeline_zb(S, M, f, b, [0] * S, c) == oracle_mod.pipeline(S, M, f, b, c)


def test_in_flight(oracle_mod):
    """A forward's activations stay until its W: walking the op lists gives at most S, and
    exactly min(S, M) on every stage -- the peak 1F1B has on its first stage only."""
    for S in range(1, 9):
        for M in range(1, 3 * S + 2):
            for s in range(S):
                live = peak = 0
                for kind, _ in brute_sim.zb_op_list(S, M, s):
                    live += kind == "F"
                    live -= kind == "W"
                    peak = max(peak, live)
                assert oracle_mod.in_flight_zb(S, M, s) == peak == min(S, M)


def _plan(n):
    return dict(hdr=np.zeros(n, np.uint32), cut=np.zeros((16, n), np.uint8), cls=np.zeros((4, n), np.uint32),
                types=np.zeros((4, n), np.uint64))


def _set(p, i, cuts, classes, tp=1, zero=0, zb=1, overlap=0, v=1):
    p["hdr"][i] = (tp.bit_length() - 1) | ((len(cuts) // v - 1) << 4) | ((len(classes) - 1) << 8) | (
        zero << 10) | (overlap << 13) | ((v - 1) << 14) | (zb << 16)
    for s, c in enumerate(cuts):
        p["cut"][s, i] = c
    for g, (reps, nmb, tv) in enumerate(classes):
        p["cls"][g, i] = reps | (nmb << 16)
        p["types"][g, i] = tv


def test_plan_split_and_schedule(oracle_mod, workloads):
    """Dense model: W is half of each stage's backward time (rounded down; all of it is compute)
    and B the rest; the stage times
    equal the plain plan's, the ends are the zero-bubble pipeline over them, and the iteration is
    the latest end plus its sync."""
    m = workloads.model("gpt2-small")
    c = workloads.cluster_two_type_8()
    o = oracle_mod.Oracle(m, c)
    p = _plan(2)
    _set(p, 0, (3, 7, 12), ((1, 8, 0x010),))
    _set(p, 1, (3, 7, 12), ((1, 8, 0x010),), zb=0)
    d, d0 = o.detail(p, 0), o.detail(p, 1)
    assert d["f"] == d0["f"] and d["b"] == d0["b"] and d["c"] == d0["c"] and d["tdp"] == d0["tdp"]
    S = 3
    assert d["w"][0] == [x // 2 for x in d["b"][0]]
    bi = [x - y for x, y in zip(d["b"][0], d["w"][0])]
    end = oracle_mod.pipeline_zb(S, 8, d["f"][0], bi, d["w"][0], d["c"][0][:S - 1])
    assert d["end"][0] == end
    assert d["time"] == max(e + t for e, t in zip(end, d["tdp"][0]))
    assert d["time"] < d0["time"]                       # the cool-down bubble shrinks


def test_memory_counts_s_in_flight(oracle_mod, workloads):
    """Every stage keeps min(S, M) micro-batches' activations under the zero-bubble order: the
    stage bytes exceed 1F1B's by (min(S, M) - min(S - s, M)) stored-activation layers."""
    m = workloads.model("gpt2-small")
    c = workloads.cluster_two_type_8()
    o = oracle_mod.Oracle(m, c)
    p = _plan(2)
    _set(p, 0, (3, 7, 12), ((1, 8, 0x010),))
    _set(p, 1, (3, 7, 12), ((1, 8, 0x010),), zb=0)
    a, b = o.stage_mem(p, 0), o.stage_mem(p, 1)
    per = o.layer_act_bytes(1, m["mbs"][0])
    for s, ns in enumerate((3, 4, 5)):
        assert int(a[0][s]) - int(b[0][s]) == ns * per * (min(3, 8) - min(3 - s, 8))


def test_invalid_zero_bubble_plans(oracle_mod, workloads):
    m = workloads.model("gpt2-small")
    c = workloads.cluster_two_type_8()
    o = oracle_mod.Oracle(m, c)
    p = _plan(5)
    _set(p, 0, (6, 12), ((1, 8, 0x10),))                                  # valid
    _set(p, 1, (6, 12), ((1, 8, 0x10),), overlap=1)                       # no overlap with it
    _set(p, 2, (3, 6, 9, 12), ((1, 8, 0x10),), v=2)                       # no interleaving with it
    _set(p, 3, (6, 12), ((1, 8, 0x10),))
    p["hdr"][3] |= np.uint32(1 << 17)                                      # reserved
    _set(p, 4, (12,), ((1, 8, 0x0),))                                     # one stage: valid
    t = o.eval(p)
    assert t[0] != MAXU and t[4] != MAXU
    assert all(t[i] == MAXU for i in (1, 2, 3)), t
    h = workloads.as_per_class(workloads.plans(workloads.workload(1), 0, 16))
    h["hdr"] |= np.uint32(1 << 16)                                        # the per-class layout does not take it
    assert np.all(o.eval(h) == MAXU)


def _moe_zb_setup(oracle_mod, workloads):
    """A Mixtral-shaped 4-layer MoE model at uniform expert load on two 4-device nodes of one
    type: two stages of 4 replicas at EP 4 (each stage's EP group fills one node, so its
    all-to-all runs on the node fabric), 4 micro-batches per replica; the hop between the stages
    crosses nodes over 25 GB/s NICs with 1000 ps per NIC side and no PCIe delay."""
    m = workloads.model("mixtral-8x7b", L=4, seq=256, global_batch=16)
    m["load_q16"] = np.full((4, 8), 65536 // 8, dtype=np.uint32)
    c = workloads.cluster_two_type_8()
    c["types"][0].update(n_nodes=2, dev_per_node=4, intra_MBps=25_000, intra_alpha_ps=1000, nic_MBps=25_000,
                         nic_alpha_ps=1000, pcie_alpha_ps=0)
    o = oracle_mod.Oracle(m, c)
    p = _plan(2)
    hdr = 2 << 2                                                  # EP 4
    _set(p, 0, (2, 4), ((4, 16, 0x00),))
    _set(p, 1, (2, 4), ((4, 16, 0x00),), zb=0)
    p["hdr"][:] |= np.uint32(hdr)
    return o, p, m, c


def test_moe_split_keeps_all_to_all_in_input_gradient(oracle_mod, workloads):
    """ZB-H1 splits a layer's backward compute into the input-gradient and the weight-gradient
    GEMMs; the MoE all-to-all of the backward pass carries input gradients between EP ranks, so it
    belongs to B.  Hand computation: per stage, Bc = the layers' (and embedding's or head's)
    backward compute, EPB = 2 all-to-alls per layer, each (ep-1) alpha + (ep-1)/ep T topk h e at
    40 ps/B (25 GB/s; the pairwise-exchange closed form), W = floor(Bc / 2), B = Bc - W + EPB.
    The hop between the stages crosses nodes: both NIC sides' 1000 ps and the activation T h e at
    40 ps/B.  The stage ends are then an event-driven replay of the zero-bubble op lists
    (independent code) over (F, B, W) and that hop, and the iteration the latest end plus the
    stage's sync.  Rejects: W taken as
    half of the whole backward including the all-to-all; the all-to-all moved into W."""
    o, p, _, _ = _moe_zb_setup(oracle_mod, workloads)
    ep, T, h, e, topk = 4, 256, 4096, 2, 2
    per_a2a = (ep - 1) * 1000 + (ep - 1) * T * topk * h * e // ep * 40
    d = o.detail(p, 0)
    assert d is not None and d["S"] == 2 and d["M"][0] == 4
    lay = [(o.layer_time(0, 1, 1, ep, l), o.layer_time(0, 1, 1, ep, l, True)) for l in range(4)]
    fc = [lay[0][0] + lay[1][0] + o.embed_time(0, 1), lay[2][0] + lay[3][0] + o.head_time(0, 1, 1)]
    bc = [lay[0][1] + lay[1][1] + o.embed_time(0, 1, True), lay[2][1] + lay[3][1] + o.head_time(0, 1, 1, True)]
    epb = 2 * 2 * per_a2a                                          # two layers per stage, two all-to-alls each
    f = [x + epb for x in fc]
    w = [x // 2 for x in bc]
    bi = [x - y + epb for x, y in zip(bc, w)]
    assert d["f"][0][:2] == f
    assert d["b"][0][:2] == [x + epb for x in bc]
    assert d["w"][0][:2] == w
    hop = 2 * 1000 + T * h * e * 40
    assert d["c"][0][0] == hop
    end = brute_sim.simulate_zb(2, 4, f, bi, w, [hop, 0])
    assert d["end"][0][:2] == end
    assert d["time"] == max(x + t for x, t in zip(end, d["tdp"][0][:2]))
    # the all-to-all really is there, and half of it is not what W holds
    assert epb > 0 and all(x != (b + epb) // 2 for x, b in zip(w, bc))
