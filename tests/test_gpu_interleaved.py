"""Parity of interleaved 1F1B (header bits 14-15 = v - 1: v model chunks per device) between
the HIP path, through the C ABI, and the oracle.  Integer picoseconds: every comparison is
bit-exact."""
import copy
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

MAXU = np.uint64(2**64 - 1)
SHAPES = [(2, 2), (2, 3), (2, 4), (3, 2), (3, 3), (3, 4), (4, 2), (4, 3), (4, 4), (5, 2), (5, 3), (6, 2), (7, 2),
          (8, 2)]


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


def _equal(got, want, what):
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, "%s: %d mismatches, first %s: gpu %d oracle %d" % (
        what, bad.size, bad[:5], int(got[bad[0]]), int(want[bad[0]]))


def _times(B, sim, p):
    return B.times_u64(sim.eval_plans(B.device_plans(p)))


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_interleaved_plans(torch, B, oracle_mod, workloads, idx):
    w = workloads.workload(idx)
    n = 40_000 + 37
    p = workloads.interleaved_plans(w, 0, n)
    say("case: interleaved plans, workload %d, %d plans" % (idx, n))
    got = _times(B, B.Sim(w["model"], w["cluster"]), p)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _equal(got, want, "interleaved workload %d" % idx)
    assert np.count_nonzero(want != MAXU) > n // 2


def _concat(a, b, order):
    out = {}
    for k in a:
        x = np.concatenate([a[k], b[k]], axis=-1)
        out[k] = np.ascontiguousarray(x[..., order])
    return out


@pytest.mark.parametrize("idx", [2, 5])
def test_interleaved_mixed_with_plain(torch, B, oracle_mod, workloads, idx):
    """Plain, overlapped and interleaved plans shuffled into one call: every kind lands in its
    own sorted range and pass."""
    w = workloads.workload(idx)
    n = 30_011
    a = workloads.plans(w, 0, n)
    a["hdr"][::7] |= np.uint32(1 << 13)
    b = workloads.interleaved_plans(w, 0, n)
    order = np.random.default_rng(idx).permutation(2 * n)
    p = _concat(a, b, order)
    say("case: plain and interleaved plans mixed, workload %d" % idx)
    got = _times(B, B.Sim(w["model"], w["cluster"]), p)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _equal(got, want, "mixed workload %d" % idx)


def _shape_case(workloads, S, v, q, n, seed):
    """The 512-device cluster with a global batch of 4 M micro-batches (M = q S), and n plans of
    one (S, v) shape: one class of 1, 2 or 4 replicas (4 M, 2 M or M micro-batches each), TP 1,
    2 or 4, random cuts and device types."""
    w = workloads.workload(3)
    m, c = dict(w["model"]), w["cluster"]
    M = q * S
    m["global_batch"] = 4 * M * m["mbs"][0]
    L, K = m["L"], len(c["types"])
    rng = np.random.default_rng(seed)
    p = dict(hdr=np.zeros(n, np.uint32), cut=np.zeros((16, n), np.uint8), cls=np.zeros((4, n), np.uint32),
             types=np.zeros((4, n), np.uint64))
    for i in range(n):
        reps = int(rng.choice([1, 2, 4]))
        cuts = np.sort(rng.choice(np.arange(1, L), S * v - 1, replace=False)).tolist() + [L]
        p["hdr"][i] = int(rng.integers(0, 3)) | ((S - 1) << 4) | (int(rng.integers(0, 2)) << 10) | ((v - 1) << 14)
        for s_, x in enumerate(cuts):
            p["cut"][s_, i] = x
        p["cls"][0, i] = reps | ((4 * M) << 16)
        p["types"][0, i] = sum(int(rng.integers(0, K)) << (4 * s_) for s_ in range(S))
    return m, c, p


@pytest.mark.parametrize("S,v", SHAPES)
def test_every_shape(torch, B, oracle_mod, workloads, S, v):
    """Every (S, v) shape from the smallest M (2S) to long schedules (256 S micro-batches per
    replica), where the steady trips are skipped once periodic."""
    for q in (2, 3, 5, 16, 64):
        m, c, p = _shape_case(workloads, S, v, q, 60, 1000 * S + 10 * v + q)
        say("case: interleaved shape S=%d v=%d q=%d" % (S, v, q))
        got = _times(B, B.Sim(m, c), p)
        want = oracle_mod.Oracle(m, c).eval(p)
        _equal(got, want, "shape %d x %d, q %d" % (S, v, q))
        assert np.count_nonzero(want != MAXU) > 40


@pytest.mark.parametrize("idx", [2, 3, 4])
def test_interleaved_stage_records(torch, B, oracle_mod, workloads, idx):
    """Per virtual stage forward/backward times, per device hops (the last one the wrap hop)
    and syncs, and the class word with v."""
    w = workloads.workload(idx)
    n = 1500
    p = workloads.interleaved_plans(w, 0, n)
    say("case: interleaved stage records workload %d" % idx)
    sim = B.Sim(w["model"], w["cluster"])
    st, cl = sim.eval_stages(B.device_plans(p))
    st = st.cpu().numpy().view(np.uint64)
    cl = cl.cpu().numpy().view(np.uint32)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    checked = 0
    for i in range(0, n, 3):
        d = o.detail(p, i)
        if d is None:
            assert np.all(cl[i] == 0)
            continue
        G = d["G"]
        S = ((int(p["hdr"][i]) >> 4) & 15) + 1
        v = ((int(p["hdr"][i]) >> 14) & 3) + 1
        for g in range(4):
            if g >= G:
                assert cl[i, g] == 0
                continue
            assert cl[i, g] == S | (G << 5) | (d["M"][g] << 8) | ((v - 1) << 24), (i, g)
            for vs in range(S * v):
                rec = [int(x) for x in st[i, g, vs]]
                want = [d["f"][g][vs], d["b"][g][vs], d["c"][g][vs] if vs < S else 0,
                        d["tdp"][g][vs] if vs < S else 0]
                assert rec == want, (idx, i, g, vs, rec, want)
        checked += 1
    assert checked > 200


@pytest.mark.parametrize("idx", [3, 4])
def test_interleaved_memory(torch, B, oracle_mod, workloads, idx):
    w = workloads.with_memory(workloads.workload(idx))
    n = 20_011
    p = workloads.interleaved_plans(w, 0, n)
    say("case: interleaved with device memory, workload %d" % idx)
    sim, o = B.Sim(w["model"], w["cluster"]), oracle_mod.Oracle(w["model"], w["cluster"])
    got = _times(B, sim, p)
    want = o.eval(p)
    _equal(got, want, "interleaved with memory, workload %d" % idx)
    assert 0 < np.count_nonzero(want != MAXU) < n
    m = 1500
    mem = sim.eval_memory(B.device_plans({k: np.ascontiguousarray(x[..., :m]) for k, x in p.items()}), m)
    mem = mem.cpu().numpy().view(np.uint64)
    for i in range(m):
        ref = o.stage_mem(p, i)
        if ref is None:
            assert np.all(mem[i] == MAXU), i
        else:
            assert np.array_equal(mem[i], ref), i


def test_interleaved_chunks_and_streams(torch, B, oracle_mod, workloads):
    """More than two 2M-plan chunks of interleaved plans (a call above 4M plans is worked in 2M
    chunks), checked on samples."""
    w = workloads.workload(3)
    n = (1 << 22) + 40_013
    p = workloads.interleaved_plans(w, 0, n)
    say("case: interleaved, %d plans in three chunks" % n)
    got = _times(B, B.Sim(w["model"], w["cluster"]), p)
    rng = np.random.default_rng(3)
    sample = np.unique(np.concatenate([rng.integers(0, n, 30_000), np.arange((1 << 21) - 50, (1 << 21) + 50), np.arange((1 << 22) - 50, (1 << 22) + 50)]))
    sub = {k: np.ascontiguousarray(x[..., sample]) for k, x in p.items()}
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(sub)
    _equal(got[sample], want, "interleaved multi-chunk")


def test_interleaved_slow_links(torch, B, oracle_mod, workloads):
    """Links slowed 40 times: hop-bound schedules that settle late or not at all."""
    w = workloads.workload(2)
    c = copy.deepcopy(w["cluster"])
    for t in c["types"]:
        t["nic_MBps"] = max(16, t["nic_MBps"] // 40)
        t["intra_MBps"] = max(16, t["intra_MBps"] // 40)
        t["pcie_MBps"] = max(16, t["pcie_MBps"] // 40) if t["pcie_MBps"] else 0
    n = 20_011
    p = workloads.random_plans_il(w["model"], c, 0x11E0 + 40, 0, n)
    say("case: interleaved, links slowed 40x, %d plans" % n)
    got = _times(B, B.Sim(w["model"], c), p)
    want = oracle_mod.Oracle(w["model"], c).eval(p)
    _equal(got, want, "interleaved links slowed 40x")


def test_interleaved_past_2_53(torch, B, oracle_mod, workloads):
    """The 4096-device cluster with devices 6 times slower: some iterations take 2^53 ps or
    more, which the fp64 pass hands to the u64 one."""
    w = workloads.workload(5)
    c = copy.deepcopy(w["cluster"])
    for t in c["types"]:
        t["tflops"] = max(1, t["tflops"] // 6)
        t["hbm_GBps"] = max(1, t["hbm_GBps"] // 6)
    n = 20_011
    p = workloads.random_plans_il(w["model"], c, 0x11E0 + 6, 0, n)
    say("case: interleaved, devices 6x slower, %d plans" % n)
    got = _times(B, B.Sim(w["model"], c), p)
    want = oracle_mod.Oracle(w["model"], c).eval(p)
    _equal(got, want, "interleaved past 2^53")
    assert np.count_nonzero((want >= 2**53) & (want != MAXU)) > 20


def test_invalid_interleaved_plans(torch, B, oracle_mod, workloads):
    """The interleaving rules (no overlap, S >= 2, S v <= 16, M a multiple of S and >= 2S, S v
    cuts ending at L, shared layout only) reject exactly as the oracle does."""
    w = workloads.workload(3)
    n = 6000
    p = workloads.interleaved_plans(w, 0, n)
    rng = np.random.default_rng(12)
    k = rng.integers(0, 6, n)
    hdr = p["hdr"].astype(np.int64)
    hdr = np.where(k == 1, hdr | (1 << 13), hdr)                                   # overlap
    hdr = np.where(k == 2, (hdr & ~(15 << 4)), hdr)                                # S = 1
    hdr = np.where(k == 3, hdr | (3 << 14), hdr)                                   # v = 4, maybe S v > 16
    p["hdr"] = hdr.astype(np.uint32)
    cls = p["cls"].astype(np.int64)
    p["cls"][0] = np.where(k == 4, (cls[0] & 0xFFFF0000) | np.maximum(1, (cls[0] & 0xFFFF) + 1), cls[0]).astype(
        np.uint32)                                                                 # M changes
    p["cut"][15] = np.where(k == 5, 1, p["cut"][15])                               # stray cut past S v
    say("case: invalid interleaved plans")
    got = _times(B, B.Sim(w["model"], w["cluster"]), p)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _equal(got, want, "invalid interleaved")
    assert np.count_nonzero(want == MAXU) > n // 3
    # the per-class layout does not take interleaving
    h = workloads.as_per_class(workloads.plans(w, 0, 64))
    h["hdr"] |= np.uint32(1 << 14)
    got = _times(B, B.Sim(w["model"], w["cluster"]), h)
    assert np.all(got == MAXU)
