"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Integer picoseconds: every comparison is bit-exact.  Small cases compare every
plan; the full-size sweeps are launched exactly as the benchmark launches them
and compared on a sample of plans (plus every plan whose time reaches 2^53 ps,
which takes the u64 path) that the oracle evaluates one by one.
"""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

MAXU = np.uint64(2**64 - 1)


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


def _sub(p, idx):
    return dict(hdr=np.ascontiguousarray(p["hdr"][idx]), cut=np.ascontiguousarray(p["cut"][:, idx]),
                cls=np.ascontiguousarray(p["cls"][:, idx]), types=np.ascontiguousarray(p["types"][:, idx]))


def _gpu_times(B, sim, p):
    dp = B.device_plans(p)
    return B.times_u64(sim.eval_plans(dp))


def _assert_equal(got, want, what):
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, "%s: %d mismatches, first %s: gpu %d oracle %d" % (
        what, bad.size, bad[:5], int(got[bad[0]]), int(want[bad[0]]))


def test_exhaustive_two_type_cluster(torch, B, oracle_mod, workloads):
    w = workloads.workload(1)
    p = workloads.plans(w)
    say("case: exhaustive 8-device, %d plans" % len(p["hdr"]))
    sim = B.Sim(w["model"], w["cluster"])
    got = _gpu_times(B, sim, p)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _assert_equal(got, want, "exhaustive")
    t = torch.from_numpy(got.view(np.int64)).cuda()
    bt, bi = B.best_tuple(sim.argmin(t))
    assert (bt, bi) == (int(want.min()), int(np.argmin(want)))


@pytest.mark.parametrize("idx", [2, 3, 4, 5])
def test_random_prefix(torch, B, oracle_mod, workloads, idx):
    w = workloads.workload(idx)
    n = 40_000 + 37                                   # several tiles and a ragged tail
    p = workloads.plans(w, 0, n)
    say("case: workload %d prefix %d" % (idx, n))
    got = _gpu_times(B, B.Sim(w["model"], w["cluster"]), p)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _assert_equal(got, want, "workload %d" % idx)
    assert np.count_nonzero(want != MAXU) > n // 2


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_stage_records(torch, B, oracle_mod, workloads, idx):
    """Per (class, stage) forward/backward/hop/DP times and micro-batch counts."""
    w = workloads.workload(idx)
    p = workloads.plans(w, 0, 1500)
    say("case: stage records workload %d" % idx)
    sim = B.Sim(w["model"], w["cluster"])
    st, cl = sim.eval_stages(B.device_plans(p))
    st = st.cpu().numpy().view(np.uint64)
    cl = cl.cpu().numpy().view(np.uint32)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    for i in range(0, 1500, 3):
        d = o.detail(p, i)
        if d is None:
            assert np.all(cl[i] == 0)
            continue
        S, G = d["S"], d["G"]
        for g in range(4):
            if g >= G:
                assert cl[i, g] == 0
                continue
            assert cl[i, g] == S | (G << 5) | (d["M"][g] << 8), (i, g)
            for s in range(S):
                rec = [int(v) for v in st[i, g, s]]
                want = [d["f"][g][s], d["b"][g][s], d["c"][g][s], d["tdp"][g][s]]
                assert rec == want, (idx, i, g, s, rec, want)


def _plan(n):
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


def test_invalid_plans(torch, B, oracle_mod, workloads):
    w = workloads.workload(1)
    p = _plan(13)
    ok = dict(cuts=(6, 12), classes=((4, 8, 0x10),))
    _set(p, 0, **ok)
    _set(p, 1, tp=8, cuts=(6, 12), classes=((1, 8, 0x10),))
    _set(p, 2, cuts=(6, 11), classes=((4, 8, 0x10),))
    _set(p, 3, cuts=(6, 6), classes=((4, 8, 0x10),))
    _set(p, 4, cuts=(6, 12), classes=((4, 7, 0x10),))
    _set(p, 5, cuts=(6, 12), classes=((4, 3, 0x10),))
    _set(p, 6, cuts=(6, 12), classes=((5, 8, 0x10),))
    _set(p, 7, cuts=(6, 12), classes=((4, 8, 0x20),))
    _set(p, 8, ep=2, cuts=(6, 12), classes=((4, 8, 0x10),))
    _set(p, 9, cuts=(6, 12), classes=((4, 8, 0x10),), mi=1)
    _set(p, 10, **ok)
    p["hdr"][10] |= 1 << 20
    _set(p, 11, cuts=(0, 12), classes=((4, 8, 0x10),))
    _set(p, 12, tp=4, cuts=(12,), classes=((1, 4, 0x0), (1, 4, 0x1)))   # valid, TP 4 fills each node
    say("case: invalid plans")
    got = _gpu_times(B, B.Sim(w["model"], w["cluster"]), p)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _assert_equal(got, want, "invalid")
    assert got[0] != MAXU and got[12] != MAXU and np.all(got[1:12] == MAXU)


def test_sizes_and_strides(torch, B, oracle_mod, workloads):
    w = workloads.workload(2)
    p = workloads.plans(w, 0, 3000)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    say("case: sizes and strides")
    for n in (1, 2, 63, 64, 65, 255, 257, 1000):
        got = B.times_u64(sim.eval_plans(dp, n=n))
        _assert_equal(got, want[:n], "n=%d" % n)
    # a window in the middle of the arrays (plane stride 3000, offset 1234)
    got = B.times_u64(sim.eval_plans(dp, n=777, offset=1234))
    _assert_equal(got, want[1234:2011], "window")
    empty = torch.zeros(0, dtype=torch.int64, device="cuda")
    sim.eval_plans(dp, n=0, out=empty)


def test_determinism(torch, B, workloads):
    w = workloads.workload(3)
    p = workloads.plans(w, 0, 300_000)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    say("case: determinism")
    a = B.times_u64(sim.eval_plans(dp)).copy()
    b = B.times_u64(sim.eval_plans(dp))
    assert np.array_equal(a, b)


def test_argmin_semantics(torch, B, workloads):
    w = workloads.workload(1)
    sim = B.Sim(w["model"], w["cluster"])
    say("case: argmin")
    inv = np.full(1000, MAXU, dtype=np.uint64)
    t = torch.from_numpy(inv.view(np.int64)).cuda()
    assert B.best_tuple(sim.argmin(t)) == (2**64 - 1, -1)
    assert B.best_tuple(sim.argmin(t, n=0)) == (2**64 - 1, -1)
    v = np.arange(5000, dtype=np.uint64)[::-1].copy() + np.uint64(7)
    v[[100, 2000, 4000]] = 3                                     # ties: lowest index wins
    v[50] = MAXU
    t = torch.from_numpy(v.view(np.int64)).cuda()
    assert B.best_tuple(sim.argmin(t, index_base=10**9)) == (3, 10**9 + 100)
    # chunks on two streams, then one reduction
    slots = torch.empty(8, dtype=torch.int64, device="cuda")
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for j in range(4):
        with torch.cuda.stream(streams[j % 2]):
            sim.argmin(t[j * 1250:(j + 1) * 1250], index_base=j * 1250, out=slots[2 * j:2 * j + 2],
                       stream=streams[j % 2])
    torch.cuda.synchronize()
    assert B.best_tuple(sim.best_reduce(slots)) == (3, 100)
    allinv = torch.from_numpy(np.array([-1, -1] * 3, dtype=np.int64)).cuda()   # {MAX, -1} slots
    assert B.best_tuple(sim.best_reduce(allinv)) == (2**64 - 1, -1)


@pytest.mark.parametrize("idx", [2, 3, 4, 5])
def test_full_size_sampled(torch, B, oracle_mod, workloads, idx):
    """Whole workload in one call (the benchmark's launch), checked on samples."""
    w = workloads.workload(idx)
    n = w["n_plans"]
    say("case: full workload %d, %d plans: generating" % (idx, n))
    p = workloads.plans(w)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    say("case: full workload %d: evaluating on GPU" % idx)
    out = sim.eval_plans(dp)
    best = B.best_tuple(sim.argmin(out))
    got = B.times_u64(out)
    rng = np.random.default_rng(idx)
    sample = np.unique(np.concatenate([rng.integers(0, n, 20_000), np.nonzero((got >= 2**53) & (got != MAXU))[0],
                                       [0, n - 1, best[1]]]))
    say("case: full workload %d: oracle on %d sampled plans (%d at or above 2^53)" % (
        idx, sample.size, int(np.count_nonzero((got >= 2**53) & (got != MAXU)))))
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(_sub(p, sample))
    _assert_equal(got[sample], want, "full workload %d" % idx)
    valid = got != MAXU
    assert best[0] == int(got[valid].min()) and best[1] == int(np.argmax(got == got[valid].min()))


def test_chunked_streams_argmin(torch, B, oracle_mod, workloads):
    """A sweep in chunks on 1, 2 and 4 streams, one argmin slot per chunk reduced on the device,
    gives the single-call result; the best plan's time matches the oracle."""
    w = workloads.workload(5)
    n, chunk = 3_000_000, 700_001
    say("case: chunked sweep of workload 5, %d plans" % n)
    p = workloads.plans(w, 0, n)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    full = sim.eval_plans(dp)
    ref = B.best_tuple(sim.argmin(full))
    chunks = [(o, min(chunk, n - o)) for o in range(0, n, chunk)]
    for ns in (1, 2, 4):
        out = torch.empty(n, dtype=torch.int64, device="cuda")
        slots = torch.empty(2 * len(chunks), dtype=torch.int64, device="cuda")
        streams = [torch.cuda.Stream() for _ in range(ns)]
        torch.cuda.synchronize()
        for j, (o, m) in enumerate(chunks):
            st = streams[j % ns]
            sim.eval_plans(dp, n=m, offset=o, out=out[o:o + m], stream=st)
            sim.argmin(out[o:o + m], index_base=o, out=slots[2 * j:2 * j + 2], stream=st)
        torch.cuda.synchronize()
        assert B.best_tuple(sim.best_reduce(slots)) == ref, ns
        assert torch.equal(out, full)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(_sub(p, np.array([ref[1]])))
    assert int(want[0]) == ref[0]


def _steady_periodic_at(S, M, f, b, c, limit):
    """First steady iteration (0-based) after which the 1F1B state has advanced
    by one constant in every component, or None within `limit` iterations."""
    out_f, last = [0] * S, [0] * S
    for m in range(min(S - 1, M)):
        for s in range(S - 1 - m):
            st = last[0] if s == 0 else max(last[s], out_f[s - 1] + c[s - 1])
            out_f[s] = st + f[s]
            last[s] = out_f[s]
    prev = None
    for i in range(min(M - (S - 1), limit)):
        for s in range(S - 1, -1, -1):
            st = last[0] if s == 0 else max(last[s], out_f[s - 1] + c[s - 1])
            out_f[s] = st + f[s]
            last[s] = (out_f[s] if s == S - 1 else max(out_f[s], last[s + 1] + c[s])) + b[s]
        x = out_f[:S - 1] + last
        if prev is not None and len({u - v for u, v in zip(x, prev)}) == 1:
            return i
        prev = x
    return None


@pytest.mark.parametrize("slow", [1, 40, 200])
def test_link_bound_schedules(torch, B, oracle_mod, workloads, slow):
    """Plans whose pipeline hops dominate (NICs and fabrics slowed `slow` times):
    many schedules never settle into a one-iteration period, so the evaluator's
    deferred full-loop pass carries a large share of the pipelines."""
    import copy
    w = workloads.workload(2)
    c = copy.deepcopy(w["cluster"])
    for t in c["types"]:
        t["nic_MBps"] = max(16, t["nic_MBps"] // slow)
        t["intra_MBps"] = max(16, t["intra_MBps"] // slow)
    n = 30_011
    p = workloads.random_plans(w["model"], c, 0x5107 + slow, 0, n)
    say("case: workload 2 model, links slowed %dx, %d plans" % (slow, n))
    got = _gpu_times(B, B.Sim(w["model"], c), p)
    o = oracle_mod.Oracle(w["model"], c)
    want = o.eval(p)
    _assert_equal(got, want, "links slowed %dx" % slow)
    assert np.count_nonzero(want != MAXU) > n // 2
    if slow == 200:
        # the case does reach pipelines that stay aperiodic past the shortcut's budget
        aperiodic = 0
        for i in range(300):
            d = o.detail(p, i)
            if d is None:
                continue
            for g in range(d["G"]):
                if d["M"][g] - (d["S"] - 1) > 40 and _steady_periodic_at(
                        d["S"], d["M"][g], d["f"][g], d["b"][g], d["c"][g], 34) is None:
                    aperiodic += 1
        say("  aperiodic pipelines in the first 300 plans: %d" % aperiodic)
        assert aperiodic > 0


def test_concurrent_multichunk_calls(torch, B, workloads):
    """Calls of several internal chunks (their deferred passes overlap on the
    context's second stream) issued concurrently on two streams of one
    context give the results of the same calls made one at a time."""
    w = workloads.workload(3)
    n = 4_500_001                                     # three internal chunks, the last ragged
    p = workloads.plans(w, 1_000_000, n)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    say("case: workload 3, two concurrent calls of %d plans" % n)
    ref = sim.eval_plans(dp)
    torch.cuda.synchronize()
    outs = [torch.empty(n, dtype=torch.int64, device="cuda") for _ in range(2)]
    streams = [torch.cuda.Stream() for _ in range(2)]
    for k in range(2):
        sim.eval_plans(dp, out=outs[k], stream=streams[k])
    torch.cuda.synchronize()
    for k in range(2):
        assert torch.equal(outs[k], ref), k


def test_tables_in_device_memory(torch, B, oracle_mod, workloads):
    """A context whose setup tables exceed the LDS budget (16 device types,
    200 layers, 4 micro-batch sizes: 0.8 MB of layer prefix sums) reads them
    from device memory; every plan still matches the oracle."""
    m = dict(workloads.workload(2)["model"])
    m["L"], m["mbs"] = 200, [1, 2, 4, 8]
    c = workloads.cluster_random(9, [2] * 16, dpn=8, jitter=True)
    n = 20_011
    p = workloads.random_plans(m, c, 0x7AB1E, 0, n)
    say("case: 16 types, 200 layers, tables in device memory, %d plans" % n)
    got = _gpu_times(B, B.Sim(m, c), p)
    want = oracle_mod.Oracle(m, c).eval(p)
    _assert_equal(got, want, "tables in device memory")
    assert np.count_nonzero(want != MAXU) > n // 2
