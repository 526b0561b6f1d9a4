"""Parity of the zero-bubble pipeline order (header bit 16: backward split into input- and
weight-gradient passes, each stage's weight passes trailing its input passes by the stage
index) between the HIP path, through the C ABI, and the oracle.  Integer picoseconds: every
comparison is bit-exact."""
import copy
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

MAXU = np.uint64(2**64 - 1)
ZB = np.uint32(1 << 16)


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


def _zb(p):
    q = {k: v.copy() for k, v in p.items()}
    q["hdr"] |= ZB
    return q


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_zero_bubble_plans(torch, B, oracle_mod, workloads, idx):
    w = workloads.workload(idx)
    n = 40_000 + 37
    p = _zb(workloads.plans(w, 0, n))
    say("case: zero-bubble plans, workload %d, %d plans" % (idx, n))
    got = _times(B, B.Sim(w["model"], w["cluster"]), p)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _equal(got, want, "zero-bubble workload %d" % idx)
    assert np.count_nonzero(want != MAXU) > n // 4
    if w["model"].get("experts"):
        # MoE plans whose backward carries an all-to-all (EP > 1) are among those compared
        ep_gt1 = ((p["hdr"] >> 2) & 3) > 0
        assert np.count_nonzero(ep_gt1 & (want != MAXU)) > n // 10


def test_zero_bubble_moe_hand_worked(torch, B, oracle_mod, workloads):
    """The hand-worked MoE plan of the oracle's pins (EP 4, uniform loads, all-to-all on the node
    fabric, weight-gradient pass half of the backward compute) and its 1F1B twin."""
    import test_oracle_zb as Z
    o, p, m, c = Z._moe_zb_setup(oracle_mod, workloads)
    say("case: hand-worked MoE zero-bubble plan")
    got = _times(B, B.Sim(m, c), p)
    want = o.eval(p)
    _equal(got, want, "hand-worked MoE zero-bubble")
    assert np.all(want != MAXU) and want[0] < want[1]


def test_zero_bubble_mixed(torch, B, oracle_mod, workloads):
    """Plain, overlapped, zero-bubble and interleaved plans in one call."""
    w = workloads.workload(2)
    n = 30_011
    p = workloads.plans(w, 0, n)
    p["hdr"][1::3] |= np.uint32(1 << 13)
    p["hdr"][2::3] |= ZB
    q = workloads.interleaved_plans(w, 0, n)
    order = np.random.default_rng(16).permutation(2 * n)
    mixed = {k: np.ascontiguousarray(np.concatenate([p[k], q[k]], axis=-1)[..., order]) for k in p}
    say("case: plain, overlapped, zero-bubble and interleaved plans mixed")
    got = _times(B, B.Sim(w["model"], w["cluster"]), mixed)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(mixed)
    _equal(got, want, "mixed kinds")


@pytest.mark.parametrize("idx", [3, 4])
def test_zero_bubble_memory(torch, B, oracle_mod, workloads, idx):
    """Every stage keeps min(S, M) micro-batches' activations: capacities reject more plans
    than under 1F1B, exactly as the oracle does; the per-device bytes match."""
    w = workloads.with_memory(workloads.workload(idx))
    n = 20_011
    p = _zb(workloads.plans(w, 0, n))
    say("case: zero-bubble with device memory, workload %d" % idx)
    sim, o = B.Sim(w["model"], w["cluster"]), oracle_mod.Oracle(w["model"], w["cluster"])
    got = _times(B, sim, p)
    want = o.eval(p)
    _equal(got, want, "zero-bubble with memory, workload %d" % idx)
    m = 1500
    mem = sim.eval_memory(B.device_plans({k: np.ascontiguousarray(x[..., :m]) for k, x in p.items()}), m)
    mem = mem.cpu().numpy().view(np.uint64)
    for i in range(m):
        ref = o.stage_mem(p, i)
        if ref is None:
            assert np.all(mem[i] == MAXU), i
        else:
            assert np.array_equal(mem[i], ref), i


def test_zero_bubble_chunks(torch, B, oracle_mod, workloads):
    w = workloads.workload(3)
    n = (1 << 21) + 30_011
    p = _zb(workloads.plans(w, 0, n))
    say("case: zero-bubble, %d plans in two chunks" % n)
    got = _times(B, B.Sim(w["model"], w["cluster"]), p)
    rng = np.random.default_rng(7)
    sample = np.unique(np.concatenate([rng.integers(0, n, 30_000), np.arange((1 << 21) - 50, (1 << 21) + 50)]))
    sub = {k: np.ascontiguousarray(x[..., sample]) for k, x in p.items()}
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(sub)
    _equal(got[sample], want, "zero-bubble multi-chunk")


def test_zero_bubble_slow_links_and_past_2_53(torch, B, oracle_mod, workloads):
    """Hop-bound schedules (links 200x slower), and devices 6x slower on the 4096-device
    cluster, where some iterations take 2^53 ps or more and are redone in u64."""
    w = workloads.workload(2)
    c = copy.deepcopy(w["cluster"])
    for t in c["types"]:
        t["nic_MBps"] = max(16, t["nic_MBps"] // 200)
        t["intra_MBps"] = max(16, t["intra_MBps"] // 200)
    n = 30_011
    p = _zb(workloads.random_plans(w["model"], c, 0x2B00, 0, n))
    say("case: zero-bubble, links slowed 200x")
    _equal(_times(B, B.Sim(w["model"], c), p), oracle_mod.Oracle(w["model"], c).eval(p), "zero-bubble slow links")
    w5 = workloads.workload(5)
    c5 = copy.deepcopy(w5["cluster"])
    for t in c5["types"]:
        t["tflops"] = max(1, t["tflops"] // 6)
        t["hbm_GBps"] = max(1, t["hbm_GBps"] // 6)
    p5 = _zb(workloads.random_plans(w5["model"], c5, 0x2B05, 0, n))
    say("case: zero-bubble, devices 6x slower")
    want = oracle_mod.Oracle(w5["model"], c5).eval(p5)
    _equal(_times(B, B.Sim(w5["model"], c5), p5), want, "zero-bubble past 2^53")
    assert np.count_nonzero((want >= 2**53) & (want != MAXU)) > 0


def test_invalid_zero_bubble_plans(torch, B, oracle_mod, workloads):
    w = workloads.workload(3)
    n = 4000
    p = workloads.plans(w, 0, n)
    k = np.random.default_rng(17).integers(0, 4, n)
    hdr = p["hdr"].astype(np.int64) | (1 << 16)
    hdr = np.where(k == 1, hdr | (1 << 13), hdr)          # with overlap
    hdr = np.where(k == 2, hdr | (1 << 14), hdr)          # with interleaving
    hdr = np.where(k == 3, hdr | (1 << 17), hdr)          # reserved
    p["hdr"] = hdr.astype(np.uint32)
    say("case: invalid zero-bubble plans")
    got = _times(B, B.Sim(w["model"], w["cluster"]), p)
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    _equal(got, want, "invalid zero-bubble")
    assert np.all(want[k > 0] == MAXU)
    h = workloads.as_per_class(workloads.plans(w, 0, 64))
    h["hdr"] |= ZB
    assert np.all(_times(B, B.Sim(w["model"], w["cluster"]), h) == MAXU)
