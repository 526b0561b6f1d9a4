"""Parity over seeded random configurations, between the HIP path, through the C ABI, and the
oracle.  Bit-exact.

Each case draws a model (the five shapes, with fresh expert loads for the MoE one; or, in
`test_random_model`, a random transformer shape), a cluster
of 1-6 device types with 1-8 nodes each, 1, 2, 4 or 8 devices per node, jittered links or not,
types whose node fabric is PCIe only, mixed latency multipliers, each of the four cluster
options on or off, device memory or none, and a global batch; then plain, overlapped,
zero-bubble, interleaved and per-class-layout plans for it.
"""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

OPTIONS = ("rail_only", "ccl_tree", "contention", "ccl_hier")
MODELS = ("gpt2-small", "llama-7b", "llama-70b", "mixtral-8x7b", "gpt3-175b")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch():
    import torch as T
    if not T.cuda.is_available():
        pytest.skip("no GPU")
    return T


@pytest.fixture(scope="module")
def B():
    from paper_2508_05370_amd import binding
    return binding


def _config(workloads, seed):
    rng = np.random.default_rng(0xC0F16000 + seed)
    name = MODELS[rng.integers(0, len(MODELS))]
    m = workloads.model(name)
    if m["experts"]:
        m["load_q16"] = workloads.dirichlet_q16(m["L"], m["experts"], seed=int(rng.integers(1, 1 << 30)))
    K = int(rng.integers(1, 7))
    nodes = [int(rng.integers(1, 9)) for _ in range(K)]
    dpn = int(rng.choice([1, 2, 4, 8]))
    c = workloads.cluster_random(int(rng.integers(0, 1000)), nodes, dpn=dpn, jitter=bool(rng.integers(0, 2)),
                                 pcie_only_types=tuple(k for k in range(K) if rng.integers(0, 4) == 0),
                                 alpha_mult=bool(rng.integers(0, 2)))
    for k, on in zip(OPTIONS, rng.integers(0, 2, len(OPTIONS))):
        c[k] = bool(on)
    if rng.integers(0, 2):
        for t in c["types"]:
            t["mem_bytes"] = int(workloads.MEM_GIB[rng.integers(0, len(workloads.MEM_GIB))]) << 30
    m["global_batch"] = int(rng.choice([8, 64, 512, 1024]))
    return name, m, c, int(rng.integers(0, 1 << 30))


@pytest.mark.parametrize("seed", range(48))
def test_random_configuration(torch, B, oracle_mod, workloads, seed):
    name, m, c, s0 = _config(workloads, seed)
    n = 4001
    p = workloads.random_plans(m, c, s0, 0, n)
    kinds = {"plain": p}
    for kind, bit in (("overlap", 13), ("zero-bubble", 16)):
        q = {k: v.copy() for k, v in p.items()}
        q["hdr"] |= np.uint32(1 << bit)
        kinds[kind] = q
    kinds["interleaved"] = workloads.random_plans_il(m, c, s0 + 1, 0, n)
    kinds["per-class"] = workloads.random_plans_het(m, c, s0 + 2, 0, n)
    sim, o = B.Sim(m, c), oracle_mod.Oracle(m, c)
    opts = ",".join(k for k in OPTIONS if c[k]) or "none"
    for kind, q in kinds.items():
        say("case: random configuration %d (%s, %d types, options %s), %s plans" % (
            seed, name, len(c["types"]), opts, kind))
        got = B.times_u64(sim.eval_plans(B.device_plans(q)))
        want = o.eval(q)
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, "configuration %d %s: %d mismatches, first %s: gpu %d oracle %d" % (
            seed, kind, bad.size, bad[:5], int(got[bad[0]]), int(want[bad[0]]))


@pytest.mark.parametrize("seed", range(48))
def test_random_configuration_records(torch, B, oracle_mod, workloads, seed):
    """Stage records (forward, backward, hop and sync per class and stage; per virtual stage for
    interleaved plans) and per-stage device memory of every class against the oracle's detail."""
    name, m, c, s0 = _config(workloads, seed)
    n = 600
    p = workloads.random_plans(m, c, s0, 0, n)
    kinds = {"plain": p}
    for kind, bit in (("overlap", 13), ("zero-bubble", 16)):
        q = {k: v.copy() for k, v in p.items()}
        q["hdr"] |= np.uint32(1 << bit)
        kinds[kind] = q
    kinds["interleaved"] = workloads.random_plans_il(m, c, s0 + 1, 0, n)
    kinds["per-class"] = workloads.random_plans_het(m, c, s0 + 2, 0, n)
    sim, o = B.Sim(m, c), oracle_mod.Oracle(m, c)
    for kind, q in kinds.items():
        say("case: random configuration %d (%s), %s stage records and memory" % (seed, name, kind))
        dq = B.device_plans(q)
        st, cl = sim.eval_stages(dq)
        st = st.cpu().numpy().view(np.uint64)
        mem = sim.eval_memory(dq, n).cpu().numpy().view(np.uint64)
        for i in range(0, n, 7):
            ref = o.stage_mem(q, i)
            if ref is None:
                assert np.all(mem[i] == np.uint64(2**64 - 1)), (seed, kind, i)
            else:
                assert np.array_equal(mem[i], ref), (seed, kind, i)
            d = o.detail(q, i)
            if d is None:
                continue
            v = ((int(q["hdr"][i]) >> 14) & 3) + 1
            for g in range(d["G"]):
                S = d["S_class"][g] if v == 1 else ((int(q["hdr"][i]) >> 4) & 15) + 1   # devices
                for vs in range(S * v):
                    rec = [int(x) for x in st[i, g, vs]]
                    want = [d["f"][g][vs], d["b"][g][vs], d["c"][g][vs] if vs < S else 0,
                            d["tdp"][g][vs] if vs < S else 0]
                    assert rec == want, (seed, kind, i, g, vs, rec, want)


def _random_model(workloads, rng):
    """A transformer shape drawn at random: depth, width, heads and grouped KV heads, MLP width
    and gating, vocabulary, positions, sequence length, micro-batch size, gradient and
    optimizer-state bytes, and for a third of them experts with top-k routing."""
    heads = int(rng.choice([4, 8, 12, 16, 32, 64, 96]))
    h = heads * int(rng.choice([64, 80, 128]))
    kvs = [k for k in range(1, heads + 1) if heads % k == 0]
    seq = int(rng.choice([512, 1024, 2048, 4096, 8192]))
    mbs = int(rng.choice([1, 2, 4]))
    m = dict(workloads.model("gpt2-small"), L=int(rng.integers(2, 97)), h=h, heads=heads,
             kv_heads=int(rng.choice(kvs)), ffn=64 * int(rng.integers(h // 64, 4 * h // 64 + 1)),
             gated=int(rng.integers(0, 2)), vocab=int(rng.integers(1000, 200_000)),
             learned_pos=seq if rng.integers(0, 2) else 0, seq=seq, mbs=[mbs],
             global_batch=mbs * int(rng.choice([8, 32, 128, 512])), grad_bytes=int(rng.choice([2, 4])),
             opt_bytes=int(rng.choice([0, 8, 12, 16])))
    if rng.integers(0, 3) == 0:
        m["experts"] = int(rng.choice([4, 8, 16]))
        m["topk"] = int(rng.integers(1, 3))
        m["expert_ffn"] = 64 * int(rng.integers(h // 64, 4 * h // 64 + 1))
        m["ffn"] = 0
        m["load_q16"] = workloads.dirichlet_q16(m["L"], m["experts"], seed=int(rng.integers(1, 1 << 30)))
    return m


@pytest.mark.parametrize("seed", range(32))
def test_random_model(torch, B, oracle_mod, workloads, seed):
    """Random model shapes on random clusters (with their options and memory): times of every
    plan kind, then stage records and device memory on sampled plans."""
    _, _, c, s0 = _config(workloads, 1000 + seed)
    m = _random_model(workloads, np.random.default_rng(0x30DE1000 + seed))
    n = 3001
    p = workloads.random_plans(m, c, s0, 0, n)
    kinds = {"plain": p}
    for kind, bit in (("overlap", 13), ("zero-bubble", 16)):
        q = {k: v.copy() for k, v in p.items()}
        q["hdr"] |= np.uint32(1 << bit)
        kinds[kind] = q
    kinds["interleaved"] = workloads.random_plans_il(m, c, s0 + 1, 0, n)
    kinds["per-class"] = workloads.random_plans_het(m, c, s0 + 2, 0, n)
    sim, o = B.Sim(m, c), oracle_mod.Oracle(m, c)
    for kind, q in kinds.items():
        say("case: random model %d (L %d, h %d, experts %d), %s plans" % (seed, m["L"], m["h"], m["experts"], kind))
        dq = B.device_plans(q)
        got = B.times_u64(sim.eval_plans(dq))
        want = o.eval(q)
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, "model %d %s: %d mismatches, first %s: gpu %d oracle %d" % (
            seed, kind, bad.size, bad[:5], int(got[bad[0]]), int(want[bad[0]]))
        mem = sim.eval_memory(dq, n).cpu().numpy().view(np.uint64)
        for i in range(0, n, 29):
            ref = o.stage_mem(q, i)
            if ref is None:
                assert np.all(mem[i] == np.uint64(2**64 - 1)), (seed, kind, i)
            else:
                assert np.array_equal(mem[i], ref), (seed, kind, i)


def _with_mbs(p, mbs, rng):
    """Move each plan to a random micro-batch size of the list where every class's micro-batch
    count divides and still gives each replica one: the count shrinks by the size, so the
    global batch stays the same (header bits 11-12 = the size's index).  Per-class-layout plans
    move each class on its own (class byte bits 6-7), so their classes mix micro-batch sizes."""
    p = {k: v.copy() for k, v in p.items()}
    n = p["hdr"].shape[0]
    G = ((p["hdr"] >> 8) & 3) + 1
    het = "chdr" in p
    moved = 0
    for i in range(n):
        cls = [(int(p["cls"][g, i]) & 0xFFFF, int(p["cls"][g, i]) >> 16) for g in range(int(G[i]))]
        if het:
            any_moved = False
            for g, (reps, nmb) in enumerate(cls):
                j = int(rng.integers(0, len(mbs)))
                if j == 0 or nmb % mbs[j] or nmb // mbs[j] < reps:
                    continue
                p["cls"][g, i] = reps | ((nmb // mbs[j]) << 16)
                p["chdr"][i] = (int(p["chdr"][i]) & ~(3 << (8 * g + 6))) | (j << (8 * g + 6))
                any_moved = True
            moved += any_moved
            continue
        j = int(rng.integers(0, len(mbs)))
        if j == 0 or any(nmb % mbs[j] or nmb // mbs[j] < reps for reps, nmb in cls):
            continue
        for g, (reps, nmb) in enumerate(cls):
            p["cls"][g, i] = reps | ((nmb // mbs[j]) << 16)
        p["hdr"][i] = (int(p["hdr"][i]) & ~(3 << 11)) | (j << 11)
        moved += 1
    return p, moved


@pytest.mark.parametrize("seed", range(12))
def test_random_micro_batch_sizes(torch, B, oracle_mod, workloads, seed):
    """Models with four micro-batch sizes; plans of every kind moved to a random one of them,
    times and device memory."""
    _, _, c, s0 = _config(workloads, 2000 + seed)
    rng = np.random.default_rng(0x3B500000 + seed)
    m = _random_model(workloads, rng)
    m["mbs"] = [1, 2, 4, 8]
    m["global_batch"] = int(rng.choice([64, 256, 1024]))
    n = 3001
    p = workloads.random_plans(m, c, s0, 0, n)
    kinds = {"plain": p}
    for kind, bit in (("overlap", 13), ("zero-bubble", 16)):
        q = {k: v.copy() for k, v in p.items()}
        q["hdr"] |= np.uint32(1 << bit)
        kinds[kind] = q
    kinds["interleaved"] = workloads.random_plans_il(m, c, s0 + 1, 0, n)
    kinds["per-class"] = workloads.random_plans_het(m, c, s0 + 2, 0, n)
    sim, o = B.Sim(m, c), oracle_mod.Oracle(m, c)
    for kind, q0 in kinds.items():
        q, moved = _with_mbs(q0, m["mbs"], rng)
        assert moved > n // 4
        say("case: micro-batch sizes %d, %s plans (%d moved)" % (seed, kind, moved))
        dq = B.device_plans(q)
        got = B.times_u64(sim.eval_plans(dq))
        want = o.eval(q)
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, "mbs %d %s: %d mismatches, first %s: gpu %d oracle %d" % (
            seed, kind, bad.size, bad[:5], int(got[bad[0]]), int(want[bad[0]]))
        mem = sim.eval_memory(dq, n).cpu().numpy().view(np.uint64)
        for i in range(0, n, 31):
            ref = o.stage_mem(q, i)
            if ref is None:
                assert np.all(mem[i] == np.uint64(2**64 - 1)), (seed, kind, i)
            else:
                assert np.array_equal(mem[i], ref), (seed, kind, i)
