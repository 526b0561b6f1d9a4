"""Parity of the gradient-sync/backward overlap (header bit 13) between the HIP path, through
the C ABI, and the oracle.  Integer picoseconds: every comparison is bit-exact."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

MAXU = np.uint64(2**64 - 1)
OVERLAP = np.uint32(1 << 13)


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
def test_overlap_plans(torch, B, oracle_mod, workloads, idx):
    """Every other plan overlaps, so waves mix both kinds of sync."""
    w = workloads.workload(idx)
    n = min(40_000 + 37, w["n_plans"])
    p = workloads.plans(w, 0, n)
    p["hdr"][::2] |= OVERLAP
    say("case: overlap, workload %d, %d plans" % (idx, n))
    sim = B.Sim(w["model"], w["cluster"])
    got = B.times_u64(sim.eval_plans(B.device_plans(p)))
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _equal(got, want, "overlap workload %d" % idx)
    q = {k: v.copy() for k, v in p.items()}
    q["hdr"] &= ~OVERLAP
    plain = oracle_mod.Oracle(w["model"], w["cluster"]).eval(q)
    assert np.count_nonzero(want[::2] != plain[::2]) > 0


@pytest.mark.parametrize("idx", [2, 4])
def test_overlap_stage_records(torch, B, oracle_mod, workloads, idx):
    """The sync each stage leaves after its last backward pass."""
    w = workloads.workload(idx)
    n = 1500
    p = workloads.plans(w, 0, n)
    p["hdr"] |= OVERLAP
    say("case: overlap stage records workload %d" % idx)
    st, cl = B.Sim(w["model"], w["cluster"]).eval_stages(B.device_plans(p))
    st = st.cpu().numpy().view(np.uint64)
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    for i in range(0, n, 3):
        d = o.detail(p, i)
        if d is None:
            continue
        for g in range(d["G"]):
            for s in range(d["S"]):
                assert int(st[i, g, s, 3]) == d["tdp"][g][s], (idx, i, g, s)


def test_overlap_with_device_memory_and_chunks(torch, B, oracle_mod, workloads):
    """Overlap plans over more than two 2M-plan chunks, with device memory checked."""
    w = workloads.with_memory(workloads.workload(2), [48, 80, 32])
    n = (1 << 22) + 20_011
    p = workloads.plans(w, 0, n)
    p["hdr"] |= OVERLAP
    say("case: overlap with memory, %d plans in three chunks" % n)
    got = B.times_u64(B.Sim(w["model"], w["cluster"]).eval_plans(B.device_plans(p)))
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _equal(got, want, "overlap with memory")
    assert 0 < np.count_nonzero(want != MAXU) < n


def test_overlap_rejected_with_per_class_layout(torch, B, workloads):
    w = workloads.workload(3)
    p = workloads.het_plans(w, 0, 4096)
    p["hdr"] |= OVERLAP
    got = B.times_u64(B.Sim(w["model"], w["cluster"]).eval_plans(B.device_plans(p)))
    assert np.all(got == MAXU)


def test_overlap_without_dp(torch, B, oracle_mod, workloads):
    """One 8-stage replica holding every micro-batch: a DP group of one, no gradient sync, so
    overlap changes nothing.  Every placement of 4 type-A and 4 type-B stages."""
    import itertools
    w = workloads.workload(1)
    pats = [sum(1 << (4 * s) for s in c) for c in itertools.combinations(range(8), 4)]
    n = len(pats)
    q = dict(hdr=np.full(n, 7 << 4, np.uint32), cut=np.zeros((16, n), np.uint8), cls=np.zeros((4, n), np.uint32),
             types=np.zeros((4, n), np.uint64))
    q["cls"][0, :] = 1 | (8 << 16)
    for s, v in enumerate([1, 2, 3, 4, 6, 8, 10, 12]):
        q["cut"][s, :] = v
    q["types"][0, :] = np.array(pats, dtype=np.uint64)
    sim = B.Sim(w["model"], w["cluster"])
    a = B.times_u64(sim.eval_plans(B.device_plans(q)))
    q2 = {k: v.copy() for k, v in q.items()}
    q2["hdr"] |= OVERLAP
    b = B.times_u64(sim.eval_plans(B.device_plans(q2)))
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(q2)
    assert np.all(want != MAXU)
    _equal(b, want, "overlap without DP")
    _equal(b, a, "overlap without DP equals no overlap")
