"""Every plan of workloads 2-5 against the oracle, and the exact argmin.

The HIP path evaluates each sweep as the benchmark does (one call over the whole 1M-, 16M- and
4M-plan sweeps; the 64M-plan GPT-3-shaped sweep in 4M-plan chunks on two streams with one argmin
slot per chunk reduced on the device).  The oracle evaluates every plan on the host's CPU share
(16 threads at most).  Every u64 time must match bit for bit, and the (time, index) minimum must be
the oracle's lowest-index minimum.  These are the long GPU tests (about two minutes in all, most
of it the oracle), so they sort after the others.
"""
import os
import sys
import time

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

MAXU = np.uint64(2**64 - 1)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def host_threads():
    """Oracle threads: the CPUs this process may run on, at most 16 (one GPU's share of a box)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


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


def _oracle_argmin(t):
    """Lowest index of the minimum time (-1 and the sentinel when every plan is invalid)."""
    i = int(np.argmin(t))
    return (int(t[i]), i) if t[i] != MAXU else (int(MAXU), -1)


def _compare(got, want, what):
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, "%s: %d of %d plans differ, first %s: gpu %d oracle %d" % (
        what, bad.size, got.size, bad[:5], int(got[bad[0]]), int(want[bad[0]]))


@pytest.mark.parametrize("idx", [2, 3, 4])
def test_full_sweep_one_call(torch, B, oracle_mod, workloads, idx):
    w = workloads.workload(idx)
    n = w["n_plans"]
    say("case: full sweep of workload %d (%s), %d plans, one call" % (idx, w["name"], n))
    p = workloads.plans(w, 0, n)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    out = sim.eval_plans(dp)
    best = B.best_tuple(sim.argmin(out))
    got = B.times_u64(out)
    del dp, out
    torch.cuda.synchronize()
    t0 = time.time()
    want = oracle_mod.Oracle(w["model"], w["cluster"]).eval(p, nthreads=host_threads())
    say("  oracle: %d plans in %.1f s on %d threads" % (n, time.time() - t0, host_threads()))
    _compare(got, want, "workload %d" % idx)
    assert best == _oracle_argmin(want), (best, _oracle_argmin(want))
    say("  0 mismatches; argmin plan %d at %d ps" % (best[1], best[0]))


def test_full_sweep_chunked_streams(torch, B, oracle_mod, workloads):
    """Workload 5: 64M plans in 16 chunks of 4M.  All chunks are launched before any is checked,
    their evaluations and argmins alternating over two streams (concurrent calls on one context),
    then one device reduction of the 16 argmin slots; the oracle checks every chunk."""
    w = workloads.workload(5)
    n, ch = w["n_plans"], 1 << 22
    assert n == 16 * ch
    sim = B.Sim(w["model"], w["cluster"])
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    say("case: full sweep of workload 5 (%s): generating %d plans" % (w["name"], n))
    p = workloads.plans(w, 0, n)
    dp = B.device_plans(p)
    out = torch.empty(n, dtype=torch.int64, device="cuda")
    slots = torch.empty(2 * (n // ch), dtype=torch.int64, device="cuda")
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    main = torch.cuda.current_stream()
    ev = main.record_event()
    say("case: workload 5, 16 chunks launched on two streams")
    for j, off in enumerate(range(0, n, ch)):
        st = streams[j % 2]
        st.wait_event(ev)
        sim.eval_plans(dp, n=ch, offset=off, out=out[off:off + ch], stream=st)
        sim.argmin(out[off:off + ch], index_base=off, out=slots[2 * j:2 * j + 2], stream=st)
    for st in streams:
        main.wait_stream(st)
    best = B.best_tuple(sim.best_reduce(slots))
    got = B.times_u64(out)
    del dp, out
    best_t, best_i = int(MAXU), -1
    t0 = time.time()
    for j, off in enumerate(range(0, n, ch)):
        sub = {k: (v[off:off + ch] if k == "hdr" else np.ascontiguousarray(v[:, off:off + ch])) for k, v in p.items()}
        want = o.eval(sub, nthreads=host_threads())
        _compare(got[off:off + ch], want, "workload 5 chunk %d" % j)
        t, i = _oracle_argmin(want)
        if i >= 0 and (t < best_t or (t == best_t and off + i < best_i)):
            best_t, best_i = t, off + i
        say("  chunk %d of 16 checked (%.1f s of oracle so far)" % (j, time.time() - t0))
    assert best == (best_t, best_i), (best, (best_t, best_i))
    say("  0 mismatches over %d plans; argmin plan %d at %d ps" % (n, best_i, best_t))
