"""Resumable chunked sweep over the plans of a seeded workload.

Plans are regenerated chunk by chunk from (seed, plan index), so a sweep of any size needs one
chunk of host and device memory at a time.  After every chunk the state -- the next chunk and the
best (time, index) so far -- is written to a JSON file (replaced atomically), and a sweep started
with an existing state file resumes at its next chunk.  Ties between chunks go to the lower plan
index, so a resumed sweep ends with exactly the argmin of an uninterrupted one.
"""
import json
import os

MAXU = (1 << 64) - 1


def _better(a, b):
    """Lexicographic (time, index) order; index -1 = no valid plan."""
    if b[1] < 0:
        return a
    if a[1] < 0:
        return b
    return min(a, b)


def load_state(path, w, chunk):
    """The saved state for workload w and this chunk size, or a fresh one."""
    fresh = {"workload": w["name"], "n_plans": w["n_plans"], "chunk": chunk, "next_chunk": 0,
             "best": [MAXU, -1], "chunks_done": 0}
    if not path or not os.path.exists(path):
        return fresh
    with open(path) as f:
        st = json.load(f)
    for k in ("workload", "n_plans", "chunk"):
        if st.get(k) != fresh[k]:
            raise ValueError("state file %s is for %s=%r, not %r" % (path, k, st.get(k), fresh[k]))
    return st


def save_state(path, st):
    tmp = path + ".tmp"
    with open(tmp, "w") as f:
        json.dump(st, f)
        f.flush()
        os.fsync(f.fileno())
    os.replace(tmp, path)


def run(w, evaluate, chunk=1 << 22, state_path=None, stop_after=None, plans_fn=None):
    """Sweep every plan of workload w in chunks of `chunk`.

    evaluate(plans, index_base) -> (time, index): the best plan of one chunk (index in the whole
    sweep, -1 if none is valid).  plans_fn(w, first, n) generates a chunk (default: the workload
    generator).  stop_after: return after this many chunks of this call (the state says where to
    go on).  Returns the state: next_chunk, chunks_done and best = [time, index].
    """
    if plans_fn is None:
        from . import workloads
        plans_fn = workloads.plans
    st = load_state(state_path, w, chunk)
    n = w["n_plans"]
    nchunks = -(-n // chunk)
    done_here = 0
    while st["next_chunk"] < nchunks:
        if stop_after is not None and done_here >= stop_after:
            break
        j = st["next_chunk"]
        off = j * chunk
        m = min(chunk, n - off)
        t, i = evaluate(plans_fn(w, off, m), off)
        st["best"] = list(_better(tuple(st["best"]), (int(t), int(i))))
        st["next_chunk"] = j + 1
        st["chunks_done"] = st.get("chunks_done", 0) + 1
        done_here += 1
        if state_path:
            save_state(state_path, st)
    return st


def gpu_evaluator(sim, stream=None):
    """evaluate() for run(): one sim_eval_plans call and one sim_argmin per chunk on `stream`,
    synchronised before it returns (the state must not run ahead of the device)."""
    import torch
    from . import binding as B

    def evaluate(plans, index_base):
        n = plans["hdr"].shape[0]
        dp = B.device_plans(plans)
        out = sim.eval_plans(dp, n=n, stream=stream)
        slot = sim.argmin(out, index_base=index_base, stream=stream)
        (torch.cuda.current_stream() if stream is None else stream).synchronize()
        return B.best_tuple(slot)
    return evaluate
