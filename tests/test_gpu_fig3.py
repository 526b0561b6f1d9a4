"""GPU parity on Sec. 3's worked example (Fig. 3) in the form the per-class layout expresses
(tests/test_oracle_fig3.py works it by hand): two classes at TP 2 and TP 1 with different layer
splits over 4 H100 + 4 A100, batches 16 and 8, with equal and with different micro-batch sizes;
also with every cluster option on, and with the devices' memory (the 70B model does not fit, so
the plan is invalid).  Times and stage records equal the oracle's."""
import sys

import numpy as np
import pytest

from test_oracle_fig3 import _plans

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


@pytest.mark.parametrize("options", [(), ("contention",), ("rail_only", "ccl_tree", "contention")])
def test_fig3_plans(torch, oracle_mod, workloads, options):
    from paper_2508_05370_amd import binding as B
    m = workloads.model("llama-70b", global_batch=24, mbs=[1, 2])
    c = dict(workloads.cluster_fig3(), **{k: True for k in options})
    p0, p1 = _plans(False), _plans(True)
    p = {k: np.ascontiguousarray(np.concatenate([p0[k], p1[k]], axis=-1)) for k in p0}
    say("case: Fig. 3 example, options %s" % (",".join(options) or "none"))
    sim, o = B.Sim(m, c), oracle_mod.Oracle(m, c)
    dp = B.device_plans(p)
    got = B.times_u64(sim.eval_plans(dp))
    want = o.eval(p)
    assert np.all(want != MAXU)
    assert np.array_equal(got, want), (got, want)
    st, cl = sim.eval_stages(dp)
    st = st.cpu().numpy().view(np.uint64)
    for i in range(2):
        d = o.detail(p, i)
        for g in range(2):
            S = len(d["f"][g])
            assert int(cl[i, g]) & 31 == S
            assert [int(x) for x in st[i, g, :S, 0]] == d["f"][g]
            assert [int(x) for x in st[i, g, :S, 1]] == d["b"][g]
            assert [int(x) for x in st[i, g, :S - 1, 2]] == d["c"][g][:S - 1]
            assert [int(x) for x in st[i, g, :S, 3]] == d["tdp"][g]


def test_fig3_memory_and_header_rules(torch, oracle_mod, workloads):
    from paper_2508_05370_amd import binding as B
    m = workloads.model("llama-70b", global_batch=24, mbs=[1, 2])
    c = workloads.cluster_fig3()
    for t, gib in zip(c["types"], (80, 40)):
        t["mem_bytes"] = gib << 30
    p = _plans(True)
    q = {k: v.copy() for k, v in p.items()}
    q["hdr"][0] |= 1 << 11                    # the header's micro-batch field is unused in this layout
    both = {k: np.ascontiguousarray(np.concatenate([p[k], q[k]], axis=-1)) for k in p}
    got = B.times_u64(B.Sim(m, c).eval_plans(B.device_plans(both)))
    assert np.array_equal(got, oracle_mod.Oracle(m, c).eval(both))
    assert np.all(got == MAXU)
    mem = B.Sim(m, c).eval_memory(B.device_plans(p)).cpu().numpy().view(np.uint64)
    assert np.array_equal(mem[0], oracle_mod.Oracle(m, c).stage_mem(p, 0))
