"""Pins of the oracle's device-memory feasibility check (peak bytes per device).

Parallelism exists to fit the model in device memory (Sec. 2) and device types
differ in it (Sec. 3 example, Table 5: A100 40 GB, H100 80 GB); the paper gives
no memory formula, so the pins are a published activation count, the 1F1B
schedule itself, and invariants of the parameter accounting.
"""
import numpy as np
import pytest

from oracle import brute_sim

MAXU = np.uint64(2**64 - 1)


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


@pytest.mark.parametrize("name,tps", [("gpt2-small", (1, 2, 4)), ("gpt3-175b", (1, 2, 4, 8))])
def test_stored_activations_match_korthikanti(oracle_mod, workloads, name, tps):
    """Korthikanti et al. 2022 ("Reducing Activation Recomputation in Large Transformer
    Models", Sec. 4.1-4.2): a GPT layer with 2-byte activations and tensor parallelism t
    stores s b h (10 + 24/t + 5 a s / (h t)) bytes.  Of these, 2 s b h are the two one-byte
    dropout masks after the attention projection and after the MLP, and 5 a s^2 b / t the
    attention scores, their softmax and its dropout (mask and output).  Without dropout and
    with a fused attention kernel that recomputes the scores, the rest is what the oracle
    counts."""
    m = workloads.model(name)
    o = oracle_mod.Oracle(m, workloads.cluster_two_type_8())
    s, h, a = m["seq"], m["h"], m["heads"]
    for t in tps:
        for b in (1, 2, 3):
            korthikanti = s * b * h * 10 + s * b * h * 24 // t + 5 * a * s * s * b // t
            masks = 2 * s * b * h
            scores = 5 * a * s * s * b // t
            assert o.layer_act_bytes(t, b) == korthikanti - masks - scores, (name, t, b)


def test_one_expert_top1_moe_is_a_gated_dense_layer_plus_router(oracle_mod, workloads):
    """An MoE layer with one expert and top-1 routing sends every token through one gated
    MLP of the expert width: it stores what the gated dense layer of that width stores, plus
    the router's input."""
    dense = workloads.model("llama-7b")
    moe = workloads.model("llama-7b", ffn=0, experts=1, topk=1, expert_ffn=dense["ffn"],
                          load_q16=np.full((dense["L"], 1), 65536, np.uint32))
    c = workloads.cluster_two_type_8()
    od, om = oracle_mod.Oracle(dense, c), oracle_mod.Oracle(moe, c)
    for t in (1, 2, 4):
        for b in (1, 2):
            router_in = b * dense["seq"] * dense["h"] * dense["dtype_bytes"]
            assert om.layer_act_bytes(t, b) == od.layer_act_bytes(t, b) + router_in


def test_in_flight_follows_the_schedule(oracle_mod):
    """The micro-batches a stage holds at once, counted by walking the 1F1B op order of the
    independent event simulator (a forward adds one, a backward frees one)."""
    for S in range(1, 9):
        for M in range(1, 13):
            for s in range(S):
                live = peak = 0
                for kind, _ in brute_sim.op_list(S, M, s):
                    live += 1 if kind == "F" else -1
                    peak = max(peak, live)
                assert oracle_mod.in_flight(S, M, s) == peak, (S, M, s)


def _mem_cluster(workloads, gib=None):
    c = workloads.cluster_two_type_8()
    if gib is not None:
        for t, g in zip(c["types"], gib):
            t["mem_bytes"] = g << 30
    return c


def _state(o, p, i, m):
    """Per-stage bytes without activations: a plan with one micro-batch per replica keeps
    one micro-batch in flight on every stage."""
    mem = o.stage_mem(p, i)
    cuts = [0] + [int(v) for v in p["cut"][:, i] if v]
    return [int(mem[0, s]) - (cuts[s + 1] - cuts[s]) * o.layer_act_bytes(1, m["mbs"][0])
            for s in range(len(cuts) - 1)]


def test_state_bytes_sum_to_the_model(oracle_mod, workloads):
    """At TP 1 without ZeRO, the stages of any layer split together hold every parameter once,
    each with weight, gradient and optimizer bytes (parameter counts pinned to Table 6 and the
    published model sizes in test_oracle_pins)."""
    m = workloads.model("gpt2-small")
    o = oracle_mod.Oracle(m, _mem_cluster(workloads))
    per = m["param_bytes"] + m["grad_bytes"] + m["opt_bytes"]
    total = per * o.param_count(with_head=True)
    for cuts in ((12,), (5, 12), (1, 2, 12), (3, 6, 9, 12), tuple(range(1, 13))):
        p = _plan()
        _set(p, 0, cuts=cuts, classes=((1, 8, 0),))
        p["cls"][0, 0] = 1 | (1 << 16)            # one micro-batch: one in flight everywhere
        w = dict(m, global_batch=1)
        c = _mem_cluster(workloads)
        c["types"][0]["n_nodes"] = 4              # 16 devices: room for 12 single-device stages
        o1 = oracle_mod.Oracle(w, c)
        assert sum(_state(o1, p, 0, w)) == total, cuts


def test_zero_splits_only_the_optimizer(oracle_mod, workloads):
    """ZeRO with one replica changes nothing.  With d replicas, each stage's optimizer state
    (opt_bytes per parameter of the stage, counts pinned in test_oracle_pins) shrinks to its
    share rounded up; weights, gradients and activations stay."""
    m = workloads.model("gpt2-small")
    o = oracle_mod.Oracle(m, _mem_cluster(workloads))
    p = _plan(4)
    _set(p, 0, cuts=(6, 12), classes=((1, 8, 0x10),), zero=0)
    _set(p, 1, cuts=(6, 12), classes=((1, 8, 0x10),), zero=1)
    _set(p, 2, cuts=(6, 12), classes=((4, 8, 0x10),), zero=0)
    _set(p, 3, cuts=(6, 12), classes=((4, 8, 0x10),), zero=1)
    m0, m1, m2, m3 = (o.stage_mem(p, i) for i in range(4))
    assert np.array_equal(m0, m1)
    assert np.array_equal(m0, m2)        # replicas alone do not change a device's bytes
    embed = o.param_count(with_head=False) - o.rank_params(1, 1, 12)
    head = o.param_count(with_head=True) - o.param_count(with_head=False)
    for s, P in enumerate((o.rank_params(1, 1, 6) + embed, o.rank_params(1, 1, 6) + head)):
        opt = m["opt_bytes"] * P
        assert int(m2[0, s]) - int(m3[0, s]) == opt - -(-opt // 4), s


def test_capacity_boundary(oracle_mod, workloads):
    """A plan fits exactly when every device's peak bytes are within its type's capacity; a
    fitting plan's time does not depend on the capacities."""
    m = workloads.model("llama-7b", global_batch=8, seq=1024)
    c0 = _mem_cluster(workloads)
    o0 = oracle_mod.Oracle(m, c0)
    p = _plan(3)
    _set(p, 0, tp=2, cuts=(16, 32), classes=((2, 8, 0x10),))             # 4 A then 4 B devices
    _set(p, 1, tp=2, cuts=(10, 32), classes=((1, 4, 0x01), (1, 4, 0x10)), zero=1)
    _set(p, 2, tp=1, cuts=(32,), classes=((4, 4, 0x0), (4, 4, 0x1)))
    t0 = o0.eval(p)
    assert np.all(t0 != MAXU)
    for i in range(3):
        mem = o0.stage_mem(p, i)
        S = ((int(p["hdr"][i]) >> 4) & 15) + 1
        G = ((int(p["hdr"][i]) >> 8) & 3) + 1
        need = [0, 0]
        for g in range(G):
            for s in range(S):
                k = (int(p["types"][g, i]) >> (4 * s)) & 15
                need[k] = max(need[k], int(mem[g, s]))
        for k in range(2):
            if need[k] == 0:
                continue
            for delta, fits in ((0, True), (-1, False)):
                c = workloads.cluster_two_type_8()
                c["types"][0]["mem_bytes"] = need[0] if k == 0 else 1 << 50
                c["types"][1]["mem_bytes"] = need[1] if k == 1 else 1 << 50
                c["types"][k]["mem_bytes"] += delta
                got = oracle_mod.Oracle(m, c).eval(p)[i]
                assert (got == t0[i]) if fits else (got == MAXU), (i, k, delta)


def test_memory_of_invalid_and_absent(oracle_mod, workloads):
    w = workloads.workload(1)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    p = _plan(2)
    _set(p, 0, cuts=(6, 12), classes=((4, 8, 0x10),))
    _set(p, 1, cuts=(6, 11), classes=((4, 8, 0x10),))                   # last cut != L
    mem = o.stage_mem(p, 0)
    assert np.all(mem[0, :2] > 0) and np.all(mem[0, 2:] == 0) and np.all(mem[1:] == 0)
    assert o.stage_mem(p, 1) is None


def test_zero_splits_expert_state_over_replicas_per_ep(oracle_mod, workloads):
    """Expert parameters are synchronised over replicas / EP (each EP rank holds its own
    experts), so ZeRO splits their optimizer state over that many devices, and the rest of the
    state over all replicas."""
    m = workloads.model("mixtral-8x7b", global_batch=8)
    m["load_q16"] = np.full((m["L"], m["experts"]), 65536 // m["experts"], np.uint32)
    o = oracle_mod.Oracle(m, _mem_cluster(workloads))
    L = m["L"]
    # experts per rank halve when EP doubles: the expert part of a layer at EP e is twice the drop
    expert = {e: 2 * (o.rank_params(1, e, 1) - o.rank_params(1, 2 * e, 1)) for e in (1, 2)}
    dense = o.rank_params(1, 1, 1) - expert[1]
    embed = o.param_count(with_head=False) - o.rank_params(1, 1, L)
    head = o.param_count(with_head=True) - o.param_count(with_head=False)
    for reps, ep in ((2, 2), (4, 2), (4, 1)):
        p = _plan(2)
        for z in (0, 1):
            _set(p, z, ep=ep, cuts=(L,), classes=((reps, 8, 0),), zero=z)
        diff = int(o.stage_mem(p, 0)[0, 0]) - int(o.stage_mem(p, 1)[0, 0])
        od = m["opt_bytes"] * (L * dense + embed + head)
        oe = m["opt_bytes"] * L * expert[ep]
        want = (od - -(-od // reps)) + (oe - -(-oe // (reps // ep)))
        assert diff == want, (reps, ep)
