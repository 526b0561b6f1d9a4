"""Parity at full size and with every cluster option at once, between the HIP path, through the
C ABI, and the oracle.  Bit-exact.

* Each plan kind the benchmark times beside the headline (overlapped gradient sync, per-class
  layout, zero-bubble order, interleaved 1F1B) on the 16M-plan Llama-70B-shaped workload in one
  call, as the benchmark launches it, checked on sampled plans: 20 000 at random, every plan at or
  above 2^53, the first, the last and the best.
* The four cluster options (rail-only forwarding, tree and two-level all-reduce, link contention)
  switched on together, over a shuffled mix of plain, overlapped, zero-bubble and interleaved
  plans in one call, and over per-class-layout plans.
"""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

MAXU = np.uint64(2**64 - 1)
ALL_FLAGS = dict(rail_only=True, ccl_tree=True, contention=True, ccl_hier=True)


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


def _sub(p, idx):
    return {k: np.ascontiguousarray(v[..., idx]) for k, v in p.items()}


def _concat(parts, order):
    return {k: np.ascontiguousarray(np.concatenate([q[k] for q in parts], axis=-1)[..., order]) for k in parts[0]}


@pytest.mark.parametrize("kind", ["overlap", "per-class", "zero-bubble", "interleaved"])
def test_benchmark_leg_full_size_sampled(torch, B, oracle_mod, workloads, kind):
    w = workloads.workload(3)
    n = w["n_plans"]
    say("case: full workload 3, %s plans, %d plans: generating" % (kind, n))
    if kind == "per-class":
        p = workloads.het_plans(w)
    elif kind == "interleaved":
        p = workloads.interleaved_plans(w)
    else:
        p = workloads.plans(w)
        p["hdr"] |= np.uint32(1 << 13 if kind == "overlap" else 1 << 16)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    say("case: full workload 3, %s plans: evaluating on GPU" % kind)
    out = sim.eval_plans(dp)
    best = B.best_tuple(sim.argmin(out))
    got = B.times_u64(out)
    del dp, out
    big = np.nonzero((got >= 2**53) & (got != MAXU))[0]
    rng = np.random.default_rng(0x1E65)
    sample = np.unique(np.concatenate([rng.integers(0, n, 20_000), big, [0, n - 1, max(best[1], 0)]]))
    say("case: full workload 3, %s plans: oracle on %d sampled plans (%d at or above 2^53)" % (
        kind, sample.size, big.size))
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(_sub(p, sample))
    _equal(got[sample], want, "full workload 3, %s" % kind)
    valid = got != MAXU
    assert np.count_nonzero(valid) > n // 2
    assert best[0] == int(got[valid].min()) and best[1] == int(np.argmax(got == got[valid].min()))


@pytest.mark.parametrize("idx", [2, 3, 4, 5])
def test_all_cluster_options_mixed_kinds(torch, B, oracle_mod, workloads, idx):
    w = workloads.workload(idx)
    c = dict(w["cluster"], **ALL_FLAGS)
    n = 12_007
    a = workloads.plans(w, 0, 3 * n)
    a["hdr"][n:2 * n] |= np.uint32(1 << 13)
    a["hdr"][2 * n:] |= np.uint32(1 << 16)
    b = workloads.interleaved_plans(w, 0, n)
    p = _concat([a, b], np.random.default_rng(idx).permutation(4 * n))
    say("case: every cluster option, plain/overlap/zero-bubble/interleaved mixed, workload %d" % idx)
    got = B.times_u64(B.Sim(w["model"], c).eval_plans(B.device_plans(p)))
    want = oracle_mod.Oracle(w["model"], c).eval(p)
    _equal(got, want, "every option, mixed kinds, workload %d" % idx)
    base = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p)
    assert np.array_equal(want == MAXU, base == MAXU)
    assert np.count_nonzero(want != base) > 100


@pytest.mark.parametrize("idx", [2, 3, 4, 5])
def test_all_cluster_options_per_class(torch, B, oracle_mod, workloads, idx):
    w = workloads.workload(idx)
    c = dict(w["cluster"], **ALL_FLAGS)
    n = 30_011
    p = workloads.het_plans(w, 0, n)
    say("case: every cluster option, per-class plans, workload %d" % idx)
    got = B.times_u64(B.Sim(w["model"], c).eval_plans(B.device_plans(p)))
    _equal(got, oracle_mod.Oracle(w["model"], c).eval(p), "every option, per-class, workload %d" % idx)


@pytest.mark.parametrize("idx", [3, 5])
@pytest.mark.parametrize("kind", ["plain", "per-class"])
def test_all_cluster_options_stage_records(torch, B, oracle_mod, workloads, idx, kind):
    """Per (class, stage) forward/backward/hop times and the sync each stage waits for, with the
    four cluster options on."""
    w = workloads.workload(idx)
    c = dict(w["cluster"], **ALL_FLAGS)
    n = 1500
    p = workloads.het_plans(w, 0, n) if kind == "per-class" else workloads.plans(w, 0, n)
    say("case: every cluster option, %s stage records, workload %d" % (kind, idx))
    st, cl = B.Sim(w["model"], c).eval_stages(B.device_plans(p))
    st = st.cpu().numpy().view(np.uint64)
    cl = cl.cpu().numpy().view(np.uint32)
    o = oracle_mod.Oracle(w["model"], c)
    checked = 0
    for i in range(0, n, 3):
        d = o.detail(p, i)
        if d is None:
            assert np.all(cl[i] == 0)
            continue
        for g in range(d["G"]):
            for s in range(d["S_class"][g]):
                rec = [int(v) for v in st[i, g, s]]
                want = [d["f"][g][s], d["b"][g][s], d["c"][g][s], d["tdp"][g][s]]
                assert rec == want, (idx, i, g, s, rec, want)
        checked += 1
    assert checked > 200


@pytest.mark.parametrize("idx", [3, 4])
def test_all_cluster_options_with_memory(torch, B, oracle_mod, workloads, idx):
    """Per-type device memory and the four cluster options together, over mixed plan kinds."""
    w = workloads.with_memory(workloads.workload(idx))
    c = dict(w["cluster"], **ALL_FLAGS)
    n = 10_007
    a = workloads.plans(w, 0, 2 * n)
    a["hdr"][n:] |= np.uint32(1 << 16)
    b = workloads.interleaved_plans(w, 0, n)
    p = _concat([a, b], np.random.default_rng(idx + 10).permutation(3 * n))
    say("case: every cluster option with device memory, workload %d" % idx)
    got = B.times_u64(B.Sim(w["model"], c).eval_plans(B.device_plans(p)))
    want = oracle_mod.Oracle(w["model"], c).eval(p)
    _equal(got, want, "every option with memory, workload %d" % idx)
    assert 0 < np.count_nonzero(want != MAXU) < 3 * n


@pytest.mark.parametrize("idx", [3, 5])
def test_all_cluster_options_two_chunks(torch, B, oracle_mod, workloads, idx):
    """More than two 2M-plan chunks in one call (a call above 4M plans is worked in 2M chunks:
    double-buffered workspaces, side streams) with every cluster option on, over mixed plan kinds;
    checked on sampled plans."""
    w = workloads.workload(idx)
    c = dict(w["cluster"], **ALL_FLAGS)
    n = (1 << 22) + 4097
    a = workloads.plans(w, 0, n)
    a["hdr"][1::5] |= np.uint32(1 << 13)
    a["hdr"][2::5] |= np.uint32(1 << 16)
    b = workloads.interleaved_plans(w, 0, n // 4)
    p = _concat([a, b], np.random.default_rng(idx + 20).permutation(n + n // 4))
    say("case: every cluster option, three chunks of mixed kinds, workload %d" % idx)
    got = B.times_u64(B.Sim(w["model"], c).eval_plans(B.device_plans(p)))
    rng = np.random.default_rng(idx + 30)
    sample = np.unique(np.concatenate([rng.integers(0, got.size, 20_000), [0, got.size - 1],
                                       np.arange((1 << 21) - 50, (1 << 21) + 50), np.arange((1 << 22) - 50, (1 << 22) + 50)]))
    want = oracle_mod.Oracle(w["model"], c).eval(_sub(p, sample))
    _equal(got[sample], want, "every option, three chunks, workload %d" % idx)
