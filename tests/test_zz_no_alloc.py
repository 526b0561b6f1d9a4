"""The allocation-free entry point (sim_eval_plans_noalloc) against sim_eval_plans.

Called through the C ABI on the same plans: two calls in a row on the library's static
workspace, the second with fewer plans (the first call's contents stay in the array), must give
the same u64 times as the allocating entry point bit for bit, in both plan layouts, with plans
of every kind (plain, overlapped, zero-bubble, interleaved).  Sizes above the documented limit
are rejected with SIM_ESIZE before any launch.
"""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


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


def _mixed(workloads, w, n):
    p = workloads.plans(w, 0, n)
    p["hdr"][1::4] |= np.uint32(1 << 13)
    p["hdr"][2::4] |= np.uint32(1 << 16)
    q = workloads.interleaved_plans(w, 0, n // 4)
    return {k: np.ascontiguousarray(np.concatenate([p[k], q[k]], axis=-1)) for k in p}


def _two_calls(torch, B, sim, p, sizes):
    """sim_eval_plans on each size, then sim_eval_plans_noalloc on each size back to back on one
    stream (the second call finds the first one's contents in the workspace)."""
    dp = B.device_plans(p)
    refs = [B.times_u64(sim.eval_plans(dp, n=n)) for n in sizes]
    outs = [torch.full((n,), -7, dtype=torch.int64, device="cuda") for n in sizes]
    torch.cuda.synchronize()
    for n, out in zip(sizes, outs):
        sim.eval_plans_noalloc(dp, n=n, out=out)
    torch.cuda.synchronize()
    return refs, [B.times_u64(o) for o in outs]


@pytest.mark.parametrize("idx", [2, 3, 4, 5])
def test_noalloc_matches_eval_plans(torch, B, workloads, idx):
    w = workloads.workload(idx)
    sim = B.Sim(w["model"], w["cluster"])
    p = _mixed(workloads, w, 240_000)
    sizes = (min(p["hdr"].shape[0], B.SIM_NOALLOC_MAX_PLANS), 30_011)
    say("case: noalloc vs eval_plans, workload %d, %s plans" % (idx, sizes))
    refs, gots = _two_calls(torch, B, sim, p, sizes)
    for n, ref, got in zip(sizes, refs, gots):
        bad = np.nonzero(ref != got)[0]
        assert bad.size == 0, (idx, n, bad[:5])
        assert np.count_nonzero(ref != np.uint64(2**64 - 1)) > n // 4


def test_noalloc_per_class_layout(torch, B, workloads):
    w = workloads.workload(3)
    sim = B.Sim(w["model"], w["cluster"])
    p = workloads.het_plans(w, 0, B.SIM_NOALLOC_MAX_PLANS_PER_CLASS)
    sizes = (B.SIM_NOALLOC_MAX_PLANS_PER_CLASS, 20_011)
    say("case: noalloc vs eval_plans, per-class layout, %s plans" % (sizes,))
    refs, gots = _two_calls(torch, B, sim, p, sizes)
    for n, ref, got in zip(sizes, refs, gots):
        assert np.array_equal(ref, got), n


def test_noalloc_rejects_oversized_calls(torch, B, workloads):
    w = workloads.workload(2)
    sim = B.Sim(w["model"], w["cluster"])
    n = B.SIM_NOALLOC_MAX_PLANS + 1
    dp = B.device_plans(workloads.plans(w, 0, n))
    out = torch.empty(n, dtype=torch.int64, device="cuda")
    say("case: noalloc rejects %d plans" % n)
    with pytest.raises(B.SimError) as e:
        sim.eval_plans_noalloc(dp, n=n, out=out)
    assert e.value.code == B.SIM_ESIZE
    h = workloads.het_plans(w, 0, B.SIM_NOALLOC_MAX_PLANS_PER_CLASS + 1)
    dh = B.device_plans(h)
    with pytest.raises(B.SimError) as e:
        sim.eval_plans_noalloc(dh, n=B.SIM_NOALLOC_MAX_PLANS_PER_CLASS + 1, out=out)
    assert e.value.code == B.SIM_ESIZE
