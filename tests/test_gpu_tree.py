"""Parity of the tree collectives (cluster flag `ccl_tree`: every DP all-reduce takes the faster
of the ring and a pipelined binary tree) between the HIP path, through the C ABI, and the
oracle.  The tree wins for small gradients over many replicas, so the cases use a narrow
GPT-2-shaped model (width 256) on the 512- and 4096-device clusters.  Bit-exact."""
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


@pytest.mark.parametrize("idx", [3, 5])
@pytest.mark.parametrize("kind", ["plain", "overlap", "zero-bubble", "interleaved", "per-class"])
def test_tree_collectives(torch, B, oracle_mod, workloads, idx, kind):
    m = workloads.model("gpt2-small", global_batch=1024, h=256, heads=4, kv_heads=4, ffn=1024)
    c = dict(workloads.workload(idx)["cluster"], ccl_tree=True)
    n = 20_011
    if kind == "interleaved":
        p = workloads.random_plans_il(m, c, 0x7EE2, 0, n)
    elif kind == "per-class":
        p = workloads.random_plans_het(m, c, 0x7EE3, 0, n)
    else:
        p = workloads.random_plans(m, c, 0x7EE0, 0, n)
        if kind == "overlap":
            p["hdr"] |= np.uint32(1 << 13)
        if kind == "zero-bubble":
            p["hdr"] |= np.uint32(1 << 16)
    say("case: tree collectives, %s plans, cluster of workload %d" % (kind, idx))
    got = _times(B, B.Sim(m, c), p)
    want = oracle_mod.Oracle(m, c).eval(p)
    _equal(got, want, "tree collectives %s, cluster %d" % (kind, idx))
    if kind == "plain":
        ring = oracle_mod.Oracle(m, dict(c, ccl_tree=False)).eval(p)
        assert np.count_nonzero(want < ring) > 500


def test_tree_collectives_7b(torch, B, oracle_mod, workloads):
    m = workloads.model("llama-7b", global_batch=4096)
    c = dict(workloads.workload(5)["cluster"], ccl_tree=True)
    n = 20_011
    p = workloads.random_plans(m, c, 0x7EE1, 0, n)
    say("case: tree collectives, llama-7b shape on 4096 devices")
    got = _times(B, B.Sim(m, c), p)
    _equal(got, oracle_mod.Oracle(m, c).eval(p), "tree collectives 7b")
