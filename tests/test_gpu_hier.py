"""Parity of the two-level all-reduce (cluster flag `ccl_hier`: whole-node DP groups may
reduce-scatter inside nodes, all-reduce shards across nodes and all-gather inside nodes) between
the HIP path, through the C ABI, and the oracle, for every shared-layout plan kind.  Bit-exact."""
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


@pytest.mark.parametrize("idx", [2, 3, 4, 5])
@pytest.mark.parametrize("kind", ["plain", "overlap", "zero-bubble", "interleaved"])
def test_two_level_all_reduce(torch, B, oracle_mod, workloads, idx, kind):
    w = workloads.workload(idx)
    c = dict(w["cluster"], ccl_hier=True, ccl_tree=(idx == 5))
    n = 20_011
    if kind == "interleaved":
        p = workloads.interleaved_plans(w, 0, n)
    else:
        p = workloads.plans(w, 0, n)
        if kind == "overlap":
            p["hdr"] |= np.uint32(1 << 13)
        if kind == "zero-bubble":
            p["hdr"] |= np.uint32(1 << 16)
    say("case: two-level all-reduce, %s plans, workload %d" % (kind, idx))
    got = B.times_u64(B.Sim(w["model"], c).eval_plans(B.device_plans(p)))
    want = oracle_mod.Oracle(w["model"], c).eval(p)
    _equal(got, want, "two-level %s workload %d" % (kind, idx))
    if kind == "plain" and idx == 4:
        base = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
        assert np.count_nonzero(want < base) > 1000
