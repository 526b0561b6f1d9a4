"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test names its source.  None of them re-types the oracle's formula: they use
printed values (Tables 1, 5, 6), textbook closed forms (pipeline fill/drain,
ring all-reduce, all-to-all, transformer FLOP counts), hand-worked timelines,
an independent event-driven simulator, and invariants.
"""
import os
import random

import numpy as np
import pytest

from oracle import brute_sim

GOLD = os.path.join(os.path.dirname(__file__), "golden")
MAXU = np.uint64(2**64 - 1)


def _rows(name):
    with open(os.path.join(GOLD, name)) as fh:
        return [ln.split() for ln in fh if ln.strip() and not ln.startswith("#")]


# ------------------------------------------------------------------ P1 link delays
def test_table5_delays(oracle_mod):
    """Table 5: delay = 9200*8/unidirectional Gb/s (Sec. 5).  NVLink/PCIe printed bidirectional."""
    for arch, nvl, nvl_ns, pcie, pcie_ns, nic, nic_ns in _rows("table5_delays.txt"):
        got_nvl = oracle_mod.alpha_ps(int(nvl) // 2)
        got_pcie = oracle_mod.alpha_ps(int(pcie) // 2)
        got_nic = oracle_mod.alpha_ps(int(nic))
        # the paper truncates to two decimals of a ns
        assert int(got_nvl) // 10 == round(float(nvl_ns) * 100), arch
        assert got_pcie == round(float(pcie_ns) * 1000), arch
        assert got_nic == round(float(nic_ns) * 1000), arch


def test_beta_exact_at_25GBps(oracle_mod):
    # 25,000 MB/s is exactly 40 ps per byte
    assert oracle_mod.beta_q(25_000) == 40 * 65536
    assert oracle_mod.link_time(1_000_000, oracle_mod.beta_q(25_000)) == 40_000_000
    assert oracle_mod.beta_q(0) == 0 and oracle_mod.link_time(10**12, 0) == 0


# ------------------------------------------------------------------ P2/P3 pipeline closed forms
def test_pipeline_uniform_no_comm(oracle_mod):
    """Uniform 1F1B pipeline without communication: (S + M - 1) * (f + b)."""
    rng = random.Random(1)
    for S in range(1, 9):
        for M in range(1, 13):
            f, b = rng.randint(1, 10**9), rng.randint(1, 10**9)
            end = oracle_mod.pipeline(S, M, [f] * S, [b] * S, [0] * (S - 1))
            assert max(end) == (S + M - 1) * (f + b)
            assert end[0] == max(end)        # the first stage finishes last


def test_pipeline_uniform_with_comm(oracle_mod):
    """Uniform stages with hop cost c: (S+M-1)(f+b) + 2c[(S-1) + (M-1) - ceil((M-1)/S)]
    (closed form derived for non-blocking sends; confirmed by event simulation)."""
    rng = random.Random(2)
    for S in range(1, 9):
        for M in range(1, 21):
            f, b, c = rng.randint(1, 30), rng.randint(1, 30), rng.randint(0, 30)
            end = oracle_mod.pipeline(S, M, [f] * S, [b] * S, [c] * (S - 1))
            pred = (S + M - 1) * (f + b) + 2 * c * ((S - 1) + (M - 1) - (-(-(M - 1) // S)))
            assert max(end) == pred, (S, M, f, b, c)


def test_pipeline_worked_timelines(oracle_mod):
    """Hand-worked 1F1B timelines.  S=2, M=3, f=[3,5], b=[6,10], c=[2]:
    stage 0: F0[0,3) F1[3,6) B0[22,28) F2[28,31) B1[37,43) B2[52,58)
    stage 1: F0[5,10) B0[10,20) F1[20,25) B1[25,35) F2[35,40) B2[40,50)"""
    assert oracle_mod.pipeline(2, 3, [3, 5], [6, 10], [2]) == [58, 50]
    _, trace = brute_sim.simulate(2, 3, [3, 5], [6, 10], [2])
    got = {(s, op): (a, b) for s, op, a, b in trace}
    want0 = {"F0": (0, 3), "F1": (3, 6), "B0": (22, 28), "F2": (28, 31), "B1": (37, 43), "B2": (52, 58)}
    want1 = {"F0": (5, 10), "B0": (10, 20), "F1": (20, 25), "B1": (25, 35), "F2": (35, 40), "B2": (40, 50)}
    for op, v in want0.items():
        assert got[(0, op)] == v
    for op, v in want1.items():
        assert got[(1, op)] == v
    # S=3, M=4, f=[2,4,3], b=[4,8,6], c=[1,3]
    assert oracle_mod.pipeline(3, 4, [2, 4, 3], [4, 8, 6], [1, 3]) == [74, 69, 58]


def test_pipeline_vs_event_simulation(oracle_mod):
    """The recurrence equals an independent time-ordered event simulation."""
    rng = random.Random(3)
    for _ in range(4000):
        S, M = rng.randint(1, 6), rng.randint(1, 10)
        f = [rng.randint(0, 40) for _ in range(S)]
        b = [rng.randint(0, 40) for _ in range(S)]
        c = [rng.randint(0, 40) for _ in range(S - 1)]
        assert oracle_mod.pipeline(S, M, f, b, c) == brute_sim.simulate(S, M, f, b, c)[0], (S, M, f, b, c)


def test_pipeline_monotone_in_M(oracle_mod):
    rng = random.Random(4)
    for _ in range(300):
        S = rng.randint(1, 8)
        f = [rng.randint(1, 50) for _ in range(S)]
        b = [rng.randint(1, 50) for _ in range(S)]
        c = [rng.randint(0, 50) for _ in range(S - 1)]
        prev = None
        for M in range(1, 15):
            end = oracle_mod.pipeline(S, M, f, b, c)
            if prev is not None:
                assert all(x >= y for x, y in zip(end, prev))
            assert end[0] == max(end)
            prev = end


# ------------------------------------------------------------------ P6 ring all-reduce
def test_ring_allreduce_closed_form(oracle_mod):
    """Ring all-reduce of B bytes over p members: 2(p-1)*alpha + 2(p-1)/p * B / bw;
    reduce-scatter + all-gather of the same bytes costs the same."""
    for p in (2, 3, 4, 8, 32, 128):
        for B in (p * 1000, p * 123457, p * 10**8):
            alpha = 368_000
            t = oracle_mod.dp_sync(p, 0, B, 0, alpha, 25_000)
            assert t == 2 * (p - 1) * alpha + 2 * (p - 1) * (B // p) * 40
            rsag = oracle_mod.dp_sync(p, 1, B, B, alpha, 25_000)
            assert rsag == t
            half = oracle_mod.dp_sync(p, 1, B, 0, alpha, 25_000)   # reduce-scatter alone
            assert half == (p - 1) * alpha + (p - 1) * (B // p) * 40 + (p - 1) * alpha
    assert oracle_mod.dp_sync(1, 0, 10**9, 10**9, 10**6, 25_000) == 0


# ------------------------------------------------------------------ P5 parameter counts
def _table6_model(workloads, row):
    name, L, h, heads, ffn, seq, maxpos, vocab, nominal = row
    m = workloads.model("gpt2-small", L=int(L), h=int(h), heads=int(heads), kv_heads=int(heads), ffn=int(ffn),
                        seq=int(seq), learned_pos=int(maxpos), vocab=int(vocab))
    return m, float(nominal)


def test_table6_parameter_counts(oracle_mod, workloads):
    """Table 6 shapes reproduce the parameter counts in the model names (GPT family ties
    the output head to the input embedding, so the head is counted once)."""
    c = workloads.cluster_two_type_8()
    for row in _rows("table6_models.txt"):
        m, nominal = _table6_model(workloads, row)
        o = oracle_mod.Oracle(m, c)
        n = o.param_count(with_head=False)
        assert abs(n / nominal - 1) < 0.02, (row[0], n)


def test_public_parameter_counts(oracle_mod, workloads):
    """GPT-2 small: 85M non-embedding parameters; Llama-2 70B (80 layers, Sec. 3): ~70B with
    grouped-query attention; Llama 7B: ~6.7B."""
    c = workloads.cluster_two_type_8()
    o = oracle_mod.Oracle(workloads.model("gpt2-small"), c)
    assert abs(o.rank_params(1, 1, 12) / 85e6 - 1) < 0.01
    o = oracle_mod.Oracle(workloads.model("llama-70b"), c)
    assert abs(o.param_count(True) / 70e9 - 1) < 0.02
    o = oracle_mod.Oracle(workloads.model("llama-7b"), c)
    assert abs(o.param_count(True) / 6.74e9 - 1) < 0.01


def test_table1_message_sizes(oracle_mod, workloads):
    """Table 1: TP/PP message = one micro-batch activation (67 MB at 1 x 4096 x 8192 bf16);
    DP message ~4.4 GB of fp32 gradients for a TP8/PP8 rank (10 of 80 layers)."""
    g = dict(r for r in _rows("table1_llama2_70b.txt"))
    o = oracle_mod.Oracle(workloads.model("llama-70b"), workloads.cluster_two_type_8())
    act = o.act_bytes(1)
    assert act == 1 * 4096 * 8192 * 2 and act // 2**20 == 64 and round(act / 1e6) == int(g["tp_pp_message_MB"])
    layers = int(g["layers"]) // int(g["pp"])
    grads = 4 * o.rank_params(int(g["tp"]), 1, layers)
    assert abs(grads / float(g["dp_message_bytes"]) - 1) < 0.05


# ------------------------------------------------------------------ transformer FLOP counts
def _compute_bound_cluster(workloads):
    c = workloads.cluster_two_type_8()
    c["types"][0]["tflops"] = 1               # 1 TFLOP/s: time in ps == FLOPs
    c["types"][0]["hbm_GBps"] = 10**15        # memory never binds (each op costs >= 1 ps)
    return c


def test_layer_flops_gpt(oracle_mod, workloads):
    """Forward FLOPs of a GPT layer (f = 4h): 24*B*s*h^2 + 4*B*s^2*h; TP divides them;
    backward is twice the forward (Narayanan et al., SC'21)."""
    m = workloads.model("gpt2-small")
    o = oracle_mod.Oracle(m, _compute_bound_cluster(workloads))
    h, s = m["h"], m["seq"]
    for b in (1, 2, 4):
        for t in (1, 2, 4):
            want = (24 * b * s * h * h + 4 * b * s * s * h) // t
            fwd = o.layer_time(0, t, b, 1, 0)
            bwd = o.layer_time(0, t, b, 1, 0, bwd=True)
            assert 0 <= fwd - want <= 8          # at most 1 ps per memory-only op
            assert 0 <= bwd - 2 * want <= 8


def test_layer_flops_llama_gqa(oracle_mod, workloads):
    """Gated MLP (3 matrices, 6*T*h*f) and grouped-query attention (K/V width kv*d)."""
    m = workloads.model("llama-70b", seq=512)
    o = oracle_mod.Oracle(m, _compute_bound_cluster(workloads))
    h, s, f, kvw = m["h"], m["seq"], m["ffn"], m["kv_heads"] * (m["h"] // m["heads"])
    T = s
    want = 2 * T * h * (h + 2 * kvw) + 4 * s * s * h + 2 * T * h * h + 6 * T * h * f
    assert 0 <= o.layer_time(0, 1, 1, 1, 0) - want <= 8
    assert 0 <= o.layer_time(0, 8, 1, 1, 0) - want // 8 <= 8


def test_head_flops(oracle_mod, workloads):
    """LM head: 2*T*h*V' with V' the vocabulary padded to a multiple of 128 (50257 -> 50304)."""
    m = workloads.model("gpt2-small")
    o = oracle_mod.Oracle(m, _compute_bound_cluster(workloads))
    T, h = m["seq"], m["h"]
    assert 0 <= o.head_time(0, 1, 1) - 2 * T * h * 50304 <= 3
    assert 0 <= o.head_time(0, 4, 1) - 2 * T * h * 50304 // 4 <= 3


def test_layer_weight_bytes_match_parameters(oracle_mod, workloads):
    """Memory-bound layer: bytes are affine in the micro-batch; the weight part equals e times
    the rank's weight matrices (the parameter count less the two norm vectors)."""
    m = workloads.model("llama-7b", seq=256)
    c = workloads.cluster_two_type_8()
    c["types"][0]["tflops"] = 10**15          # compute never binds
    c["types"][0]["hbm_GBps"] = 1000         # time in ps == bytes
    o = oracle_mod.Oracle(m, c)
    for t in (1, 2, 4):
        b1, b2, b3 = (o.layer_time(0, t, b, 1, 0) for b in (1, 2, 3))
        assert b3 - b2 == b2 - b1
        weights = b1 - (b2 - b1)
        assert weights == m["dtype_bytes"] * (o.rank_params(t, 1, 1) - 2 * m["h"])


# ------------------------------------------------------------------ whole plans
def _plan(n=1):
    return dict(hdr=np.zeros(n, np.uint32), cut=np.zeros((16, n), np.uint8), cls=np.zeros((4, n), np.uint32),
                types=np.zeros((4, n), np.uint64))


def _set(p, i, tp=1, ep=1, cuts=(12,), classes=((1, 1, 0),), zero=0, mi=0):
    pp, G = len(cuts), len(classes)
    p["hdr"][i] = (tp.bit_length() - 1) | ((ep.bit_length() - 1) << 2) | ((pp - 1) << 4) | ((G - 1) << 8) | (
        zero << 10) | (mi << 11)
    for s, v in enumerate(cuts):
        p["cut"][s, i] = v
    for g, (reps, nmb, tv) in enumerate(classes):
        p["cls"][g, i] = reps | (nmb << 16)
        p["types"][g, i] = tv


def test_zero_link_single_stage_is_sum_of_ops(oracle_mod, workloads):
    """PP=1, no links: the iteration is M micro-batches of (embedding + layers + head) fwd+bwd."""
    m = workloads.model("gpt2-small")
    c = workloads.cluster_two_type_8()
    for t in c["types"]:
        t.update(intra_MBps=0, nic_MBps=0, intra_alpha_ps=0, nic_alpha_ps=0)
    o = oracle_mod.Oracle(m, c)
    p = _plan()
    _set(p, 0, cuts=(12,), classes=((1, 8, 0),))
    one = sum(o.layer_time(0, 1, 1, 1, l) + o.layer_time(0, 1, 1, 1, l, True) for l in range(12))
    one += o.embed_time(0, 1) + o.embed_time(0, 1, True) + o.head_time(0, 1, 1) + o.head_time(0, 1, 1, True)
    assert int(o.eval(p)[0]) == 8 * one


def test_invalid_plans_are_sentinel(oracle_mod, workloads):
    w = workloads.workload(1)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    p = _plan(12)
    ok = dict(cuts=(6, 12), classes=((4, 8, 0x10),))
    _set(p, 0, **ok)                                          # valid: 4 A then 4 B
    _set(p, 1, tp=8, cuts=(6, 12), classes=((1, 8, 0x10),))   # tp 8 does not fit a 4-device node / 12 heads
    _set(p, 2, cuts=(6, 11), classes=((4, 8, 0x10),))        # last cut != L
    _set(p, 3, cuts=(6, 6), classes=((4, 8, 0x10),))         # empty stage
    _set(p, 4, cuts=(6, 12), classes=((4, 7, 0x10),))        # 7 != global batch 8
    _set(p, 5, cuts=(6, 12), classes=((4, 3, 0x10),))        # fewer micro-batches than replicas
    _set(p, 6, cuts=(6, 12), classes=((5, 8, 0x10),))        # 5 replicas exceed 4 devices
    _set(p, 7, cuts=(6, 12), classes=((4, 8, 0x20),))        # type 2 does not exist
    _set(p, 8, ep=2, cuts=(6, 12), classes=((4, 8, 0x10),))  # EP on a dense model
    _set(p, 9, cuts=(6, 12), classes=((4, 8, 0x10),), mi=1)  # micro-batch size index out of range
    _set(p, 10, **ok)
    p["hdr"][10] |= 1 << 20                                   # reserved header bit
    _set(p, 11, cuts=(0, 12), classes=((4, 8, 0x10),))       # first cut 0
    out = o.eval(p)
    assert out[0] != MAXU
    assert all(out[i] == MAXU for i in range(1, 12)), out


def test_faster_hardware_never_slower(oracle_mod, workloads):
    """Monotonicity: raising any device or link rate never increases an iteration time."""
    w = workloads.workload(2)
    p = workloads.plans(w, 0, 3000)
    base = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    for key, factor in (("tflops", 2), ("hbm_GBps", 2), ("intra_MBps", 2), ("nic_MBps", 2), ("pcie_MBps", 2)):
        for k in range(len(w["cluster"]["types"])):
            c = {**w["cluster"], "types": [dict(t) for t in w["cluster"]["types"]]}
            c["types"][k][key] *= factor
            out = oracle_mod.Oracle(w["model"], c).eval(p)
            assert np.all(out <= base), (key, k)
            if key in ("tflops", "hbm_GBps"):
                assert np.any(out < base), (key, k)


def test_class_permutation_invariance(oracle_mod, workloads):
    """Without jitter and with every class on its own nodes, the order of classes is irrelevant."""
    m = workloads.model("llama-7b")
    c = workloads.cluster_random(2, [3, 3, 2])
    o = oracle_mod.Oracle(m, c)
    p = _plan(2)
    # class 0: 8 replicas of (type0, type1) at tp 1 -> 8 devices per pool = one node each
    # class 1: 8 replicas of (type1, type0)
    a, b = (8, 256, 0x10), (8, 256, 0x01)
    _set(p, 0, cuts=(16, 32), classes=(a, b))
    _set(p, 1, cuts=(16, 32), classes=(b, a))
    out = o.eval(p)
    assert out[0] == out[1] != MAXU


def test_moe_all_to_all_closed_form(oracle_mod, workloads):
    """Uniform expert load: each all-to-all costs (ep-1)*alpha + (ep-1)/ep * T*topk*h*e / bw
    (pairwise exchange, Mixtral-shaped layer, 25 GB/s links)."""
    m = workloads.model("mixtral-8x7b", L=4, seq=256, global_batch=8)
    m["load_q16"] = np.full((4, 8), 65536 // 8, dtype=np.uint32)
    c = workloads.cluster_two_type_8()
    c["types"][0].update(n_nodes=2, dev_per_node=4, intra_MBps=25_000, intra_alpha_ps=1000)
    o = oracle_mod.Oracle(m, c)
    p = _plan()
    ep = 4
    _set(p, 0, ep=ep, cuts=(4,), classes=((8, 8, 0x0),))     # 8 replicas on two 4-device nodes: EP groups intra
    d = o.detail(p, 0)
    comp = sum(o.layer_time(0, 1, 1, ep, l) for l in range(4)) + o.embed_time(0, 1) + o.head_time(0, 1, 1)
    epf = d["f"][0][0] - comp
    T, h, e, topk = 256, 4096, 2, 2
    per_a2a = (ep - 1) * 1000 + (ep - 1) * T * topk * h * e // ep * 40
    assert epf == 2 * 4 * per_a2a


# ------------------------------------------------------------------ hand-worked communication and cost terms
def _one_type(n_nodes, dpn, **kw):
    t = dict(n_nodes=n_nodes, dev_per_node=dpn, tflops=300, hbm_GBps=2000, intra_MBps=25_000, pcie_MBps=0,
             nic_MBps=25_000, intra_alpha_ps=1000, pcie_alpha_ps=0, nic_alpha_ps=0)
    t.update(kw)
    return t


@pytest.mark.parametrize("tp", [2, 4, 8])
def test_tp_allreduce_closed_form(oracle_mod, workloads, tp):
    """TP all-reduces are exposed in the forward pass only (Table 1): two per layer (after the
    attention and after the MLP) and one for the vocabulary-parallel embedding on the first stage,
    each a ring all-reduce over the tp ranks of a node: 2(tp-1) steps of one latency and of an
    activation shard Act/tp.  On a 25 GB/s fabric (exactly 40 ps/B) with 1 us per message, a
    stage holding n layers gets nAR = 2n + [first stage] all-reduces; with 1000 ps per message,
    TPF = nAR 2(tp-1) 1000 ps + nAR 2(tp-1) (Act/tp) 40 ps.
    Rejects: (tp-1) steps instead of 2(tp-1); no embedding all-reduce; the whole activation per
    step; a TP term in the backward pass."""
    m = workloads.model("llama-7b", L=4, seq=256, global_batch=2)
    c = dict(types=[_one_type(2, 8)], nic_MBps_dev=None, intra_MBps_node=None)
    o = oracle_mod.Oracle(m, c)
    p = _plan()
    _set(p, 0, tp=tp, cuts=(1, 4), classes=((1, 2, 0x00),))
    d = o.detail(p, 0)
    act = 256 * 4096 * 2
    for s, (layers, first, last) in enumerate(((range(0, 1), 1, 0), (range(1, 4), 0, 1))):
        comp_f = sum(o.layer_time(0, tp, 1, 1, l) for l in layers)
        comp_b = sum(o.layer_time(0, tp, 1, 1, l, True) for l in layers)
        if first:
            comp_f += o.embed_time(0, 1)
            comp_b += o.embed_time(0, 1, True)
        if last:
            comp_f += o.head_time(0, tp, 1)
            comp_b += o.head_time(0, tp, 1, True)
        n_ar = 2 * len(layers) + first
        steps = n_ar * 2 * (tp - 1)
        assert d["f"][0][s] - comp_f == steps * 1000 + steps * (act // tp) * 40, (tp, s)
        assert d["b"][0][s] == comp_b, (tp, s)


def _hop_cluster(nodes_a=1, dpn_a=4):
    # Table 5's delays: A100-like type A with 2 x 287.5 ns PCIe trips, H100-like type B with
    # 2 x 143.75 ns, NIC processing 368 ns on both
    A = _one_type(nodes_a, dpn_a, intra_MBps=300_000, intra_alpha_ps=30_670, pcie_MBps=32_000,
                  pcie_alpha_ps=287_500, nic_MBps=25_000, nic_alpha_ps=368_000)
    B = _one_type(1, 4, intra_MBps=450_000, intra_alpha_ps=20_440, pcie_MBps=64_000, pcie_alpha_ps=143_750,
                  nic_MBps=50_000, nic_alpha_ps=368_000)
    return dict(types=[A, B], nic_MBps_dev=None, intra_MBps_node=None)


def test_pp_hop_inter_node_with_pcie(oracle_mod, workloads):
    """An inter-node pipeline hop goes GPU -> PCIe switch -> NIC on each end (Sec. 5: two PCIe
    trips per side) plus the NIC's processing delay (Table 5), and both ends pay; the activation
    crosses at the slowest of the two NICs and the two PCIe links.  Stage 0 on type A, stage 1 on
    type B: alpha = (2 x 287,500 + 368,000) + (2 x 143,750 + 368,000) ps.  With the NICs slower
    than PCIe the rate is A's NIC (40 ps/B); with A's PCIe link at 16 GB/s (62.5 ps/B) it is that
    link.  Rejects: latency of one end only; one PCIe trip per side; the PCIe rate ignored."""
    m = workloads.model("gpt2-small")
    act = 1024 * 768 * 2
    alpha = (2 * 287_500 + 368_000) + (2 * 143_750 + 368_000)
    for pcie_a, ps_per_byte in ((32_000, 40), (16_000, 62.5)):
        c = _hop_cluster()
        c["types"][0]["pcie_MBps"] = pcie_a
        o = oracle_mod.Oracle(m, c)
        p = _plan()
        _set(p, 0, cuts=(6, 12), classes=((4, 8, 0x10),))
        d = o.detail(p, 0)
        assert d["c"][0][0] == alpha + int(act * ps_per_byte), pcie_a


def test_pp_hop_intra_vs_inter_in_one_pool(oracle_mod, workloads):
    """Within one pool a hop is intra-node iff every replica's pair of devices shares a node:
    two replicas per stage on one 4-device node pay one node-fabric message (30.67 ns, and the
    activation at 300 GB/s with the per-byte rate rounded up in 2^-16 ps units); on 2-device
    nodes the stages sit on different nodes and the hop pays both ends' inter-node path on
    type A.  Rejects: the intra/inter decision taken per pool rather than per node."""
    m = workloads.model("gpt2-small")
    act = 1024 * 768 * 2
    bq_intra = -(-65536 * 10**6 // 300_000)                      # ps per byte in 2^-16 units, rounded up
    o = oracle_mod.Oracle(m, _hop_cluster(1, 4))
    p = _plan()
    _set(p, 0, cuts=(6, 12), classes=((2, 8, 0x00),))
    assert o.detail(p, 0)["c"][0][0] == 30_670 + -(-act * bq_intra // 65536)
    o2 = oracle_mod.Oracle(m, _hop_cluster(2, 2))
    assert o2.detail(p, 0)["c"][0][0] == 2 * (2 * 287_500 + 368_000) + act * 40


def test_expert_imbalance_takes_busiest_rank(oracle_mod, workloads):
    """R9: an MoE layer waits for its busiest EP rank.  On a device of 1 TFLOP/s (one flop per ps)
    whose memory is fast enough that no op's bytes cost more than 1 ps, an expert that receives n
    tokens costs 2 n h 2f (up and gate) + 1 (the activation) + 2 n f h (down) = 6 n h f + 1 ps
    forward.  At EP 2, rank 0 hosts experts 0-3 and rank 1 experts 4-7; expert e receives
    ceil(ep T topk q_e / 2^16) tokens of the ep T routed ones.  Moving load from rank 1 to rank 0
    changes the layer by the change of the busiest rank's sum, not of the sum or the mean over
    ranks (those stay put).  Rejects: sum or mean over ranks in place of the max."""
    L, E, h, f, seq, topk, ep = 1, 8, 64, 128, 16, 2, 2
    m = dict(L=L, h=h, heads=4, kv_heads=4, ffn=0, gated=1, vocab=128, learned_pos=0, seq=seq, dtype_bytes=2,
             global_batch=2, mbs=[1], experts=E, topk=topk, expert_ffn=f, grad_bytes=4, param_bytes=2, opt_bytes=12)
    c = dict(types=[_one_type(1, 4, tflops=1, hbm_GBps=4_000_000_000)], nic_MBps_dev=None, intra_MBps_node=None)

    def expert(n):
        return 6 * n * h * f + 1 if n else 2          # an idle expert still reads its two weight blocks

    def busiest(q):
        T = seq
        tok = [-(-ep * T * topk * int(x) // 65536) for x in q]
        return max(sum(expert(n) for n in tok[:4]), sum(expert(n) for n in tok[4:]))

    uniform = [8192] * 8
    skew = [16384, 16384, 8192, 8192, 4096, 4096, 4096, 4096]
    t = {}
    for name, q in (("uniform", uniform), ("skew", skew)):
        mm = dict(m, load_q16=np.array([q], dtype=np.uint32))
        t[name] = oracle_mod.Oracle(mm, c).layer_time(0, 1, 1, ep, 0)
    assert busiest(skew) != busiest(uniform)
    assert t["skew"] - t["uniform"] == busiest(skew) - busiest(uniform)


def test_embedding_bytes(oracle_mod, workloads):
    """The input embedding is a gather, not a GEMM: per token it reads one table row of h elements
    and writes one output row; with learned positions it also reads a position row and adds it
    (reading the partial sum and writing the result).  So it moves 2 T h e bytes (4 T h e with
    learned positions), whatever the vocabulary and the TP degree, at the memory rate:
    1000 B / hbm ps, i.e. exactly B ps at 1000 GB/s; backward twice that.  Rejects: the whole
    table read; positions not counted; compute-rate costing."""
    c = dict(types=[_one_type(1, 4, hbm_GBps=1000, tflops=1)], nic_MBps_dev=None, intra_MBps_node=None)
    for name, pos in (("gpt2-small", 1), ("llama-7b", 0)):
        for vocab in (32000, 64000):
            m = workloads.model(name, vocab=vocab, seq=512)
            o = oracle_mod.Oracle(m, c)
            for b in (1, 2):
                T = b * 512
                B = T * m["h"] * m["dtype_bytes"] * (4 if pos else 2)
                assert o.embed_time(0, b) == B, (name, vocab, b)
                assert o.embed_time(0, b, True) == 2 * B


def test_dp_ring_inter_node_latency(oracle_mod, workloads):
    """A DP ring whose members sit on several nodes crosses the inter-node path at every step:
    each step pays both ends' latency (two PCIe trips and the NIC on each side, Sec. 5 and
    Table 5) and moves its chunk at the slowest NIC or PCIe rate; inside one node it pays the node
    fabric's.  A 4-replica ring all-reduce of the whole model's fp32 gradients (PP 1, TP 1) over
    type A on two 2-device nodes: 2(p-1) steps of 2 (2 x 287,500 + 368,000) ps and of
    ceil(G/p) bytes at 40 ps/B (the 25 GB/s NIC; PCIe is 32 GB/s).  Two replicas on one node: the
    same ring on the fabric (30.67 ns, 300 GB/s).  Rejects: one end's latency per step."""
    m = workloads.model("gpt2-small")
    grads = 4 * oracle_mod.Oracle(m, _hop_cluster()).param_count(True)
    p = _plan()
    _set(p, 0, cuts=(12,), classes=((4, 8, 0x00),))
    d = oracle_mod.Oracle(m, _hop_cluster(2, 2)).detail(p, 0)
    steps = 2 * 3
    assert d["tdp"][0][0] == steps * 2 * (2 * 287_500 + 368_000) + steps * -(-grads // 4) * 40
    _set(p, 0, cuts=(12,), classes=((2, 8, 0x00),))
    d = oracle_mod.Oracle(m, _hop_cluster(1, 2)).detail(p, 0)
    bq = -(-65536 * 10**6 // 300_000)
    assert d["tdp"][0][0] == 2 * 30_670 + -(-(2 * -(-grads // 2)) * bq // 65536)
