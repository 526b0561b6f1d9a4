"""Parity of the rail-only network (cluster flag `rail_only`: cross-rail pipeline hops are
forwarded over a node's fabric first) between the HIP path, through the C ABI, and the oracle,
for every plan kind.  Integer picoseconds: every comparison is bit-exact."""
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


def _times(B, sim, p):
    return B.times_u64(sim.eval_plans(B.device_plans(p)))


def _rail(w):
    return dict(w["cluster"], rail_only=True)


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("kind", ["plain", "interleaved", "per-class", "zero-bubble", "overlap"])
def test_rail_only_plans(torch, B, oracle_mod, workloads, idx, kind):
    w = workloads.workload(idx)
    c = _rail(w)
    n = 20_011
    if kind == "interleaved":
        p = workloads.interleaved_plans(w, 0, n)
    elif kind == "per-class":
        p = workloads.het_plans(w, 0, n)
    else:
        p = workloads.plans(w, 0, min(n, w["n_plans"]))
        if kind == "zero-bubble":
            p["hdr"] |= np.uint32(1 << 16)
        if kind == "overlap":
            p["hdr"] |= np.uint32(1 << 13)
    say("case: rail-only network, %s plans, workload %d" % (kind, idx))
    got = _times(B, B.Sim(w["model"], c), p)
    o = oracle_mod.Oracle(w["model"], c)
    want = o.eval(p)
    _equal(got, want, "rail-only %s workload %d" % (kind, idx))
    if idx > 1 and kind == "plain":
        base = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
        assert np.count_nonzero(want != base) > 0


@pytest.mark.parametrize("idx", [2, 3])
def test_rail_only_stage_records(torch, B, oracle_mod, workloads, idx):
    w = workloads.workload(idx)
    c = _rail(w)
    n = 1500
    p = workloads.plans(w, 0, n)
    say("case: rail-only stage records, workload %d" % idx)
    st, cl = B.Sim(w["model"], c).eval_stages(B.device_plans(p))
    st = st.cpu().numpy().view(np.uint64)
    o = oracle_mod.Oracle(w["model"], c)
    for i in range(0, n, 5):
        d = o.detail(p, i)
        if d is None:
            continue
        for g in range(d["G"]):
            for s in range(d["S"]):
                assert int(st[i, g, s, 2]) == d["c"][g][s], (i, g, s)
