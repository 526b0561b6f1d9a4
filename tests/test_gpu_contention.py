"""Parity of link contention (cluster flag `contention`: the concurrent segment syncs of a stage
share its links) between the HIP path, through the C ABI, and the oracle, for per-class-layout
plans, alone and with tree collectives.  Bit-exact."""
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
def test_contention_per_class_plans(torch, B, oracle_mod, workloads, idx):
    w = workloads.workload(idx)
    c = dict(w["cluster"], contention=True)
    n = 20_011
    p = workloads.het_plans(w, 0, n)
    say("case: contention, per-class plans, workload %d" % idx)
    got = B.times_u64(B.Sim(w["model"], c).eval_plans(B.device_plans(p)))
    want = oracle_mod.Oracle(w["model"], c).eval(p)
    _equal(got, want, "contention workload %d" % idx)
    if idx > 1:
        base = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
        assert np.count_nonzero(want > base) > 100


def test_contention_with_tree_collectives(torch, B, oracle_mod, workloads):
    m = workloads.model("gpt2-small", global_batch=1024, h=256, heads=4, kv_heads=4, ffn=1024)
    c = dict(workloads.workload(5)["cluster"], contention=True, ccl_tree=True)
    p = workloads.random_plans_het(m, c, 0x7EE4, 0, 20_011)
    say("case: contention and tree collectives, per-class plans")
    got = B.times_u64(B.Sim(m, c).eval_plans(B.device_plans(p)))
    _equal(got, oracle_mod.Oracle(m, c).eval(p), "contention with trees")


@pytest.mark.parametrize("idx", [3, 4])
def test_contention_stage_records(torch, B, oracle_mod, workloads, idx):
    w = workloads.workload(idx)
    c = dict(w["cluster"], contention=True)
    n = 1500
    p = workloads.het_plans(w, 0, n)
    say("case: contention stage records, workload %d" % idx)
    st, cl = B.Sim(w["model"], c).eval_stages(B.device_plans(p))
    st = st.cpu().numpy().view(np.uint64)
    o = oracle_mod.Oracle(w["model"], c)
    for i in range(0, n, 3):
        d = o.detail(p, i)
        if d is None:
            continue
        for g in range(d["G"]):
            for s in range(d["S_class"][g]):
                assert int(st[i, g, s, 3]) == d["tdp"][g][s], (i, g, s)
