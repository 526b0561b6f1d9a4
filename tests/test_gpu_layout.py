"""Parity of the per-class layout (each replica class with its own TP degree, pipeline depth
and layer split, resharding before the gradient sync) between the HIP path, through the C
ABI, and the oracle.  Integer picoseconds: every comparison is bit-exact."""
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


def _equal(got, want, what):
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, "%s: %d mismatches, first %s: gpu %d oracle %d" % (
        what, bad.size, bad[:5], int(got[bad[0]]), int(want[bad[0]]))


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_per_class_plans(torch, B, oracle_mod, workloads, idx):
    w = workloads.workload(idx)
    n = 40_000 + 37
    p = workloads.het_plans(w, 0, n)
    say("case: per-class layout, workload %d, %d plans" % (idx, n))
    got = B.times_u64(B.Sim(w["model"], w["cluster"]).eval_plans(B.device_plans(p)))
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _equal(got, want, "per-class workload %d" % idx)
    assert np.count_nonzero(want != MAXU) > n // 4


@pytest.mark.parametrize("idx", [2, 3])
def test_per_class_encoding_of_shared_plans(torch, B, workloads, idx):
    w = workloads.workload(idx)
    n = 20_011
    p = workloads.plans(w, 0, n)
    say("case: shared plans in the per-class encoding, workload %d" % idx)
    sim = B.Sim(w["model"], w["cluster"])
    a = B.times_u64(sim.eval_plans(B.device_plans(p)))
    b = B.times_u64(sim.eval_plans(B.device_plans(workloads.as_per_class(p))))
    _equal(b, a, "per-class encoding")


@pytest.mark.parametrize("idx", [2, 3, 4, 5])
def test_per_class_stage_records(torch, B, oracle_mod, workloads, idx):
    """Per (class, stage) forward/backward/hop times and the sync each stage waits for."""
    w = workloads.workload(idx)
    n = 1500
    p = workloads.het_plans(w, 0, n)
    say("case: per-class stage records workload %d" % idx)
    sim = B.Sim(w["model"], w["cluster"])
    st, cl = sim.eval_stages(B.device_plans(p))
    st = st.cpu().numpy().view(np.uint64)
    cl = cl.cpu().numpy().view(np.uint32)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    for i in range(0, n, 3):
        d = o.detail(p, i)
        if d is None:
            assert np.all(cl[i] == 0)
            continue
        G = d["G"]
        for g in range(4):
            if g >= G:
                assert cl[i, g] == 0
                continue
            S = d["S_class"][g]
            assert cl[i, g] == S | (G << 5) | (d["M"][g] << 8), (i, g)
            for s in range(S):
                rec = [int(v) for v in st[i, g, s]]
                want = [d["f"][g][s], d["b"][g][s], d["c"][g][s], d["tdp"][g][s]]
                assert rec == want, (idx, i, g, s, rec, want)


@pytest.mark.parametrize("idx", [3, 4])
def test_per_class_memory(torch, B, oracle_mod, workloads, idx):
    w = workloads.with_memory(workloads.workload(idx))
    n = 20_011
    p = workloads.het_plans(w, 0, n)
    say("case: per-class layout with device memory, workload %d" % idx)
    sim, o = B.Sim(w["model"], w["cluster"]), oracle_mod.Oracle(w["model"], w["cluster"])
    got = B.times_u64(sim.eval_plans(B.device_plans(p)))
    want = o.eval(p)
    _equal(got, want, "per-class with memory, workload %d" % idx)
    assert 0 < np.count_nonzero(want != MAXU) < n
    m = 1500
    mem = sim.eval_memory(B.device_plans({k: np.ascontiguousarray(v[..., :m]) for k, v in p.items()}), m)
    mem = mem.cpu().numpy().view(np.uint64)
    for i in range(m):
        ref = o.stage_mem(p, i)
        if ref is None:
            assert np.all(mem[i] == MAXU), i
        else:
            assert np.array_equal(mem[i], ref), i


def test_per_class_chunks_and_streams(torch, B, oracle_mod, workloads):
    """More than two 2M-plan chunks (a call above 4M plans is worked in 2M chunks): the per-class
    cut rows follow every chunk's offset."""
    w = workloads.workload(3)
    n = (1 << 22) + 40_013
    p = workloads.het_plans(w, 0, n)
    say("case: per-class layout, %d plans in three chunks" % n)
    got = B.times_u64(B.Sim(w["model"], w["cluster"]).eval_plans(B.device_plans(p)))
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _equal(got, want, "per-class multi-chunk")


def test_per_class_layout_needs_its_cut_planes(torch, B, workloads):
    """A per-class header without the per-class cut planes is an argument error."""
    import ctypes as C
    w = workloads.workload(3)
    p = workloads.het_plans(w, 0, 64)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    ps = B.plans_struct(dp)
    ps.ccut = None
    out = torch.empty(64, dtype=torch.int64, device="cuda")
    rc = B.lib().sim_eval_plans(sim.h, C.byref(ps), 64, out.data_ptr(), B._stream(None))
    assert rc == B.SIM_EINVAL


def test_per_class_deep_and_wide_plans(torch, B, oracle_mod, workloads):
    """Classes of 16 stages (every class its own 16-way split), whole-node TP 8, and single-stage
    classes next to them, on the 512-device cluster."""
    w = workloads.workload(3)
    L = w["model"]["L"]
    rng = np.random.default_rng(7)
    n = 4096
    p = dict(hdr=np.zeros(n, np.uint32), cls=np.zeros((4, n), np.uint32), types=np.zeros((4, n), np.uint64),
             chdr=np.zeros(n, np.uint32), ccut=np.zeros((64, n), np.uint8))
    gbs = w["model"]["global_batch"]
    for i in range(n):
        G = int(rng.integers(1, 5))
        reps = [int(rng.integers(1, 3)) for _ in range(G)]
        left = gbs - sum(reps)
        nmb = [r for r in reps]
        nmb[0] += left
        ch = 0
        for g in range(G):
            tpl = int(rng.choice([0, 3])) if g % 2 else int(rng.integers(0, 4))
            pp = 16 if g % 2 == 0 else int(rng.choice([1, 16]))
            cuts = np.sort(rng.choice(np.arange(1, L), pp - 1, replace=False)).tolist() + [L]
            for s, v in enumerate(cuts):
                p["ccut"][g * 16 + s, i] = v
            ch |= (tpl | ((pp - 1) << 2)) << (8 * g)
            p["cls"][g, i] = reps[g] | (nmb[g] << 16)
            p["types"][g, i] = int(sum(int(rng.integers(0, 4)) << (4 * s) for s in range(pp)))
        p["chdr"][i] = ch
        p["hdr"][i] = (G - 1) << 8 | (int(rng.integers(0, 2)) << 10)
    say("case: per-class layout, 16-stage classes and TP 8, %d plans" % n)
    got = B.times_u64(B.Sim(w["model"], w["cluster"]).eval_plans(B.device_plans(p)))
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _equal(got, want, "deep and wide per-class plans")
    assert np.count_nonzero(want != MAXU) > n // 2


def test_per_class_empty_call(torch, B, workloads):
    w = workloads.workload(3)
    p = workloads.het_plans(w, 0, 16)
    sim = B.Sim(w["model"], w["cluster"])
    out = torch.full((16,), 7, dtype=torch.int64, device="cuda")
    sim.eval_plans(B.device_plans(p), n=0, out=out)
    torch.cuda.synchronize()
    assert torch.all(out == 7)


def test_per_class_chunk_without_valid_plans(torch, B, oracle_mod, workloads):
    """A per-class chunk whose plans are all invalid (a nonzero header micro-batch field): the
    plan-order sort counts no plan, the plan-level sync pass and the pipelines do nothing, and
    every time is the invalid marker.  Then valid plans again on the same context: the counters
    start from zero in every call."""
    w = workloads.workload(3)
    n = 20_000 + 11
    p = workloads.het_plans(w, 0, n)
    q = {k: v.copy() for k, v in p.items()}
    q["hdr"] |= np.uint32(1 << 11)
    sim = B.Sim(w["model"], w["cluster"])
    say("case: per-class layout, %d plans, none valid" % n)
    got = B.times_u64(sim.eval_plans(B.device_plans(q)))
    assert np.all(got == MAXU)
    _equal(got, oracle_mod.Oracle(w["model"], w["cluster"]).eval(q), "no valid per-class plan")
    say("case: per-class layout, the same plans valid, same context")
    got = B.times_u64(sim.eval_plans(B.device_plans(p)))
    _equal(got, oracle_mod.Oracle(w["model"], w["cluster"]).eval(p), "per-class after an empty order")
