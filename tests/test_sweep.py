"""Host logic of the resumable chunked sweep (paper_2508_05370_amd/sweep.py), on the CPU.

The chunk evaluator here is the oracle (test infrastructure standing in for the device); the
sweep itself only generates chunks, keeps the best (time, index) and the state file.  An
interrupted and resumed sweep must end with the argmin of an uninterrupted one, which must be the
lowest-index minimum over every plan.
"""
import json
import os

import numpy as np
import pytest

from paper_2508_05370_amd import sweep

MAXU = (1 << 64) - 1


def _oracle_evaluator(oracle_mod, w):
    o = oracle_mod.Oracle(w["model"], w["cluster"])
    calls = []

    def evaluate(plans, base):
        t = o.eval(plans)
        calls.append(base)
        i = int(np.argmin(t))
        return (int(t[i]), base + i) if t[i] != np.uint64(MAXU) else (MAXU, -1)
    return evaluate, calls


def _small(workloads, n):
    w = dict(workloads.workload(2))
    w["n_plans"] = n
    w["name"] = w["name"] + "/first-%d" % n
    return w


def test_resumed_sweep_matches_uninterrupted(oracle_mod, workloads, tmp_path):
    w = _small(workloads, 50_000)
    chunk = 8192                                   # seven chunks, the last one ragged
    ev, calls = _oracle_evaluator(oracle_mod, w)
    full = sweep.run(w, ev, chunk=chunk)
    assert full["next_chunk"] == 7 and calls == [j * chunk for j in range(7)]
    t = oracle_mod.Oracle(w["model"], w["cluster"]).eval(workloads.plans(w, 0, w["n_plans"]))
    assert full["best"] == [int(t.min()), int(np.argmin(t))]

    path = str(tmp_path / "state.json")
    ev2, calls2 = _oracle_evaluator(oracle_mod, w)
    st = sweep.run(w, ev2, chunk=chunk, state_path=path, stop_after=3)
    assert st["next_chunk"] == 3 and json.load(open(path))["next_chunk"] == 3
    st = sweep.run(w, ev2, chunk=chunk, state_path=path, stop_after=2)
    assert st["next_chunk"] == 5
    st = sweep.run(w, ev2, chunk=chunk, state_path=path)
    assert calls2 == [j * chunk for j in range(7)]      # every chunk once, in order
    assert st["best"] == full["best"] and st["chunks_done"] == 7
    assert not os.path.exists(path + ".tmp")
    # a finished sweep resumed again does nothing
    assert sweep.run(w, ev2, chunk=chunk, state_path=path) == st and len(calls2) == 7


def test_state_of_another_sweep_is_refused(oracle_mod, workloads, tmp_path):
    w = _small(workloads, 20_000)
    ev, _ = _oracle_evaluator(oracle_mod, w)
    path = str(tmp_path / "state.json")
    sweep.run(w, ev, chunk=4096, state_path=path, stop_after=1)
    with pytest.raises(ValueError):
        sweep.run(w, ev, chunk=8192, state_path=path)
    with pytest.raises(ValueError):
        sweep.run(_small(workloads, 30_000), ev, chunk=4096, state_path=path)


def test_chunks_without_valid_plans_and_ties(oracle_mod, workloads):
    """A chunk with no valid plan reports index -1 and never wins; equal times go to the lower index."""
    w = _small(workloads, 3000)
    seen = {0: (MAXU, -1), 1000: (50, 1500), 2000: (50, 2100)}
    st = sweep.run(w, lambda p, base: seen[base], chunk=1000, plans_fn=lambda w, off, m: None)
    assert st["best"] == [50, 1500]
    st = sweep.run(w, lambda p, base: (MAXU, -1), chunk=1000, plans_fn=lambda w, off, m: None)
    assert st["best"] == [MAXU, -1]
