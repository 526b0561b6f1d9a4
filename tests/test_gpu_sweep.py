"""The resumable chunked sweep on the GPU: the GPT-3-shaped workload's first 12M plans and a
ragged tail, regenerated chunk by chunk in 4M-plan chunks, interrupted after two chunks and
resumed, ends with the argmin of one call over the same plans, and the oracle gives that plan
the same time."""
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


def test_resumed_gpu_sweep(torch, oracle_mod, workloads, tmp_path):
    from paper_2508_05370_amd import binding as B
    from paper_2508_05370_amd import sweep
    w = dict(workloads.workload(5))
    w["n_plans"] = 3 * (1 << 22) + 777
    w["name"] += "/first-%d" % w["n_plans"]
    sim = B.Sim(w["model"], w["cluster"])
    say("case: resumable sweep of %s, 4M-plan chunks" % w["name"])
    p = workloads.plans(w, 0, w["n_plans"])
    ref = B.best_tuple(sim.argmin(sim.eval_plans(B.device_plans(p))))
    del p
    ev = sweep.gpu_evaluator(sim, torch.cuda.Stream())
    path = str(tmp_path / "state.json")
    st = sweep.run(w, ev, chunk=1 << 22, state_path=path, stop_after=2)
    assert st["next_chunk"] == 2
    say("  interrupted after 2 chunks, best so far %s" % (st["best"],))
    st = sweep.run(w, ev, chunk=1 << 22, state_path=path)
    assert st["next_chunk"] == 4 and st["chunks_done"] == 4
    assert tuple(st["best"]) == ref, (st["best"], ref)
    one = workloads.plans(w, ref[1], 1)
    assert int(oracle_mod.Oracle(w["model"], w["cluster"]).eval(one)[0]) == ref[0]
    say("  resumed sweep argmin plan %d at %d ps" % (ref[1], ref[0]))
