"""Sec. 3's worked example (Fig. 3) as a plan the per-class layout can express, worked by hand.

The paper's example trains Llama-2 70B (80 layers, global batch 24, micro-batch 1) on node A
(4 x H100) and node B (4 x A100): two data-parallel replicas with non-uniform batches (16 on the
faster one, 8 on the slower), device groups at different TP degrees (the paper's TP 3 next to
TP 1), more layers on the faster devices, and resharding before the gradient sync.  TP 3 does not
divide Llama-2 70B's 64 query heads, 8 KV heads or 28672-wide MLP, so the variant here keeps TP a
power of two:

  class 0 (16 micro-batches): TP 2, 2 stages: layers [0, 60) on 2 H100, [60, 80) on 2 A100
  class 1 ( 8 micro-batches): TP 1, 4 stages: [0, 25) H100, [25, 50) H100, [50, 65) A100, [65, 80) A100

and a second plan where class 1 runs micro-batches of 2 (4 of them), so that the classes also
differ in micro-batch size (the paper's first resharding condition).

Every quantity is rebuilt here from pinned pieces -- the oracle's per-layer costs, the ring
all-reduce and link-time closed forms, the event simulator of brute_sim.py -- composed by hand:
placement, hop tiers and latencies, the TP all-reduces, the layer segments and their DP rings,
the resharding gather and the gradient weighting, the pipelines and the iteration time.  The
oracle's stage records and time must equal them exactly.
"""
import numpy as np
import pytest

from oracle import brute_sim

H100, A100 = 0, 1
L = 80


def cdiv(a, b):
    return -(-a // b)


def _plans(het_mixed):
    p = dict(hdr=np.zeros(1, np.uint32), cls=np.zeros((4, 1), np.uint32), types=np.zeros((4, 1), np.uint64),
             chdr=np.zeros(1, np.uint32), ccut=np.zeros((64, 1), np.uint8))
    p["hdr"][0] = 1 << 8                                              # two classes, EP 1, no ZeRO
    mi1, nmb1 = (1, 4) if het_mixed else (0, 8)
    p["chdr"][0] = (1 | (1 << 2)) | ((0 | (3 << 2) | (mi1 << 6)) << 8)   # class 0: TP 2, PP 2; class 1: TP 1, PP 4
    for s, v in enumerate((60, 80)):
        p["ccut"][s, 0] = v
    for s, v in enumerate((25, 50, 65, 80)):
        p["ccut"][16 + s, 0] = v
    p["cls"][0, 0] = 1 | (16 << 16)
    p["cls"][1, 0] = 1 | (nmb1 << 16)
    p["types"][0, 0] = H100 | (A100 << 4)
    p["types"][1, 0] = H100 | (H100 << 4) | (A100 << 8) | (A100 << 12)
    return p


@pytest.fixture(scope="module")
def setup(oracle_mod, workloads):
    m = workloads.model("llama-70b", global_batch=24, mbs=[1, 2])
    c = workloads.cluster_fig3()
    return m, c, oracle_mod.Oracle(m, c)


def _expected(O, m, c, o, mixed):
    ty = c["types"]
    e, h = m["dtype_bytes"], m["h"]
    beta = O.beta_q

    def side(k):                       # one end of an inter-node path: two PCIe trips and the NIC
        return 2 * ty[k]["pcie_alpha_ps"] + ty[k]["nic_alpha_ps"]

    def inter_hop(k1, k2, act):
        bq = max(beta(ty[k1]["nic_MBps"]), beta(ty[k2]["nic_MBps"]), beta(ty[k1]["pcie_MBps"]),
                 beta(ty[k2]["pcie_MBps"]))
        return side(k1) + side(k2) + O.link_time(act, bq)

    def intra_hop(k, act):
        return ty[k]["intra_alpha_ps"] + O.link_time(act, beta(ty[k]["intra_MBps"]))

    # class: (TP, micro-batch size, cuts, stage types, micro-batches per replica)
    b1 = 2 if mixed else 1
    classes = [(2, 1, (60, 80), (H100, A100), 16), (1, b1, (25, 50, 65, 80), (H100, H100, A100, A100), 8 // b1)]
    # placement (pool-wise bump pointer in (class, stage) order): H100 devices 0-1 | 2 | 3, A100 0-1 | 2 | 3,
    # all four devices of a type in one node, so the hops between H100 and A100 stages are inter-node and
    # the others intra-node
    hops = []
    for tp, b, cuts, types, M in classes:
        act = b * m["seq"] * h * e
        hops.append([intra_hop(types[s], act) if types[s] == types[s + 1] else inter_hop(types[s], types[s + 1], act)
                     for s in range(len(cuts) - 1)] + [0])
    assert hops[0][0] == inter_hop(H100, A100, m["seq"] * h * e)
    # stage compute: the layers' costs, the embedding on stage 0, the head on the last stage, and at TP 2
    # the forward all-reduces (two per layer, one for the embedding) of 2 (tp - 1) steps of act / tp bytes
    fs, bs = [], []
    for tp, b, cuts, types, M in classes:
        f, bw, lo = [], [], 0
        for s, hi in enumerate(cuts):
            k = types[s]
            F = sum(o.layer_time(k, tp, b, 1, l, False) for l in range(lo, hi))
            B = sum(o.layer_time(k, tp, b, 1, l, True) for l in range(lo, hi))
            if s == 0:
                F += o.embed_time(k, b, False)
                B += o.embed_time(k, b, True)
            if s == len(cuts) - 1:
                F += o.head_time(k, tp, b, False)
                B += o.head_time(k, tp, b, True)
            if tp > 1:
                n_ar = 2 * (hi - lo) + (s == 0)
                steps = n_ar * 2 * (tp - 1)
                F += steps * ty[k]["intra_alpha_ps"] + O.link_time(steps * cdiv(b * m["seq"] * h * e, tp),
                                                                   beta(ty[k]["intra_MBps"]))
            f.append(F)
            bw.append(B)
            lo = hi
        fs.append(f)
        bs.append(bw)
    # layer segments: between consecutive cuts of either class
    bounds = [0, 25, 50, 60, 65, 80]
    Vp = cdiv(m["vocab"], 128) * 128

    def params(a, b_, tp):             # one TP rank's parameters of layers [a, b_)
        p = o.rank_params(tp, 1, b_ - a)
        if a == 0:
            p += Vp * h // tp + m["learned_pos"] * h
        if b_ == L:
            p += Vp * h // tp + h
        return p

    def holder(cuts, a):
        return next(s for s, v in enumerate(cuts) if v > a)

    tdp = [[0] * 2, [0] * 4]
    for a, b_ in zip(bounds, bounds[1:]):
        sg = [holder(cl[2], a) for cl in classes]
        ks = [cl[3][s] for cl, s in zip(classes, sg)]
        # the ring over both replicas (two members) on the coarsest layout, TP 1: inside one node when
        # both holding stages are on the same type (each type is one node), else between nodes
        if ks[0] == ks[1]:
            alpha, MBps = ty[ks[0]]["intra_alpha_ps"], ty[ks[0]]["intra_MBps"]
        else:
            alpha, MBps = max(2 * side(k) for k in ks), min(min(ty[k]["nic_MBps"], ty[k]["pcie_MBps"]) for k in ks)
        g = m["grad_bytes"] * params(a, b_, 1)
        ring = O.dp_sync(2, 0, g, m["param_bytes"] * params(a, b_, 1), alpha, MBps)
        assert ring == 2 * alpha + O.link_time(2 * cdiv(g, 2), beta(MBps))
        # before it, each class prepares its shard (the slowest counts): weighting by its share of the
        # batch when micro-batch sizes differ (one multiply per element, read + write of fp32 gradients
        # at the device's HBM rate), then, at TP 2, the gather of the TP-1 shard: one ring step of its
        # own shard on its node's fabric
        prep = 0
        for (tp, b, cuts, types, M), k in zip(classes, ks):
            n = params(a, b_, tp)
            t = 0
            if mixed:
                t += max(cdiv(n, ty[k]["tflops"]), cdiv(1000 * 2 * m["grad_bytes"] * n, ty[k]["hbm_GBps"]))
            if tp == 2:
                t += ty[k]["intra_alpha_ps"] + O.link_time(m["grad_bytes"] * n, beta(ty[k]["intra_MBps"]))
            prep = max(prep, t)
        for g_, s in enumerate(sg):
            tdp[g_][s] = max(tdp[g_][s], ring + prep)
    ends = []
    for (tp, b, cuts, types, M), f, bw, c_ in zip(classes, fs, bs, hops):
        end, _ = brute_sim.simulate(len(cuts), M, f, bw, c_)
        ends.append(end)
    T = max(ends[g][s] + tdp[g][s] for g in range(2) for s in range(len(classes[g][2])))
    return dict(f=fs, b=bs, c=hops, tdp=tdp, end=ends, time=T, M=[cl[4] for cl in classes])


@pytest.mark.parametrize("mixed", [False, True], ids=["micro-batch-1", "micro-batches-1-and-2"])
def test_fig3_worked_example(oracle_mod, setup, mixed):
    m, c, o = setup
    p = _plans(mixed)
    d = o.detail(p, 0)
    assert d is not None, "the example must be a valid plan"
    want = _expected(oracle_mod, m, c, o, mixed)
    assert d["M"] == want["M"]
    for key in ("f", "b", "c", "tdp", "end"):
        assert d[key] == want[key], key
    assert d["time"] == want["time"]
    assert o.eval(p)[0] == want["time"]


def test_fig3_weighting_only_when_sizes_differ(oracle_mod, setup):
    """The same split with equal micro-batch sizes has no weighting term; with sizes 1 and 2 every
    segment's sync grows by exactly the slower class's weighting pass (plus its gather)."""
    m, c, o = setup
    d0, d1 = o.detail(_plans(False), 0), o.detail(_plans(True), 0)
    assert all(a < b for ra, rb in zip(d0["tdp"], d1["tdp"]) for a, b in zip(ra, rb))


def test_fig3_header_micro_batch_field_unused(oracle_mod, setup):
    """In the per-class layout the micro-batch size is each class's own: a nonzero header field,
    or a class index past the model's sizes, makes the plan invalid."""
    m, c, o = setup
    p = _plans(True)
    q = {k: v.copy() for k, v in p.items()}
    q["hdr"][0] |= 1 << 11
    r = {k: v.copy() for k, v in p.items()}
    r["chdr"][0] |= 3 << 14                                           # class 1 at index 3 (model has 2 sizes)
    assert o.eval(p)[0] != np.uint64(2**64 - 1)
    assert o.eval(q)[0] == np.uint64(2**64 - 1)
    assert o.eval(r)[0] == np.uint64(2**64 - 1)
