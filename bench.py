"""Throughput of batched plan evaluation on one MI355X.

One step = the whole hot path over every plan of the workload: decode and
validate, place, stage costs, bottleneck links, collectives, the 1F1B pipeline
of every replica class, the DP sync, and the argmin over all plans.  Plans are
resident in HBM before timing starts.

Prints one JSON line.  Roofline: the evaluation is bound by VALU issue.  The
work of one call is counted from the plans themselves: every schedule node
the evaluation executes -- all nodes of the 1F1B recurrence (3 fp64 VALU
ops per node with a cross-stage input, 1 without), less those the periodic
shortcut skips, which the library counts on the device -- plus the cost model's per-stage and per-plan setup arithmetic priced
by formula.  The peak is the lower of the chip's issue rate (256 CUs x 64
lanes x 2.4 GHz) and the node probe's measured rate times 3, measured in the
same run.
"""
import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_VALU_SPEC = 256 * 64 * 2.4e9     # VALU lane-ops per second at one instruction per SIMD lane per clock
METRIC = "candidate plans evaluated/sec on 1 MI355X; % of binding roofline"
MAXU = np.uint64(2**64 - 1)

# Setup arithmetic of the cost model, priced in gfx950 VALU instructions per
# operation of the definition: u64 add/sub 2, u64 max 3, u64 x u32 product 2,
# link time ceil(bytes x beta / 2^16) with a 96-bit product 8, ceiling
# division by a run-time divisor 12, range maximum over a sparse table 4.
PRICE = dict(add=2, max=3, mul=2, link=8, cdiv=12, rmax=4)
P = PRICE
# per (pipeline, stage): stage compute (two prefix differences), the stage's
# place in its pool (one bump-pointer add), its slowest fabric and NIC
# (two range maxima), and its share of the iteration time (fp64 add + max)
STAGE = 2 * P["add"] + P["add"] + 2 * P["rmax"] + 2
# TP all-reduces of a stage (tp > 1): count x latency, bytes, link time, add into F
TP = 2 * P["mul"] + P["link"] + 2 * P["add"]
# MoE all-to-all of a stage (ep > 1): node test, count x latency, byte difference, link time, adds into F and B
EP = 3 + P["mul"] + P["add"] + P["link"] + 2 * P["add"]
# pipeline hop into stage s > 0: node test, two-sided latency, slowest of four rates, link time
HOP = 3 + P["add"] + 2 * P["max"] + P["link"]
# embedding on the first stage, head on the last: two adds each
ENDS = 4 * P["add"]
# DP sync of one stage, once per plan (the ring spans every class's replicas): gradient shard, count x latency,
# bytes, link time, add; ZeRO adds the parameter all-gather's shard, bytes, link time and add
RING = P["cdiv"] + 2 * P["mul"] + P["link"] + P["add"]
ZERO = P["cdiv"] + P["mul"] + P["link"] + P["add"]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _fields(p):
    hdr = p["hdr"].astype(np.int64)
    return dict(tp=1 << (hdr & 3), ep=1 << ((hdr >> 2) & 3), S=((hdr >> 4) & 15) + 1, G=((hdr >> 8) & 3) + 1,
                zero=(hdr >> 10) & 1)


def pipeline_ops(p, valid, per_node=3, first=1):
    """VALU ops of the whole pipeline recurrence, per plan: `per_node` per schedule node with a
    cross-stage input, `first` per node without one (3 and 1 in fp64 as the kernels run it; the
    int32 count of the same nodes is 7 and 2)."""
    f = _fields(p)
    S, G = f["S"], f["G"]
    ops = np.zeros(S.shape[0], dtype=np.int64)
    for c in range(4):
        reps = (p["cls"][c] & 0xFFFF).astype(np.int64)
        nmb = (p["cls"][c] >> 16).astype(np.int64)
        has = (G > c) & valid & (reps > 0)
        M = np.where(has, -(-nmb // np.maximum(reps, 1)), 0)
        ops += 2 * M * (per_node * (S - 1) + first)
    return ops


def setup_ops(p, valid, moe):
    """The cost model's setup arithmetic per plan (shared layout), priced as above: per class
    pipeline its stages' compute, placement, rates and iteration share, TP and EP terms, hops and
    the two ends; per plan and stage one DP sync (and the experts' ring for MoE models)."""
    f = _fields(p)
    S, G = f["S"], f["G"]
    per_pipe = S * STAGE + (S - 1) * HOP + ENDS + np.where(f["tp"] > 1, S * TP, 0)
    if moe:
        per_pipe = per_pipe + np.where(f["ep"] > 1, S * EP, 0)
    ring = RING + f["zero"] * ZERO
    per_plan = G * per_pipe + S * ring * (2 if moe else 1)
    return np.where(valid, per_plan, 0).astype(np.int64)


def host_threads():
    """Oracle threads: the CPUs this process may run on, at most 16 (one GPU's share of a box)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def input_hashes(p):
    """SHA-256 of each generated input array (its bytes in memory order)."""
    return {k: hashlib.sha256(np.ascontiguousarray(v).tobytes()).hexdigest() for k, v in sorted(p.items())}


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "eval_llama70b_16M_hbm_traffic.txt")
SQ_FILE = os.path.join(ROOT, "profiles", "eval_llama70b_16M_sq_counters.txt")
SOURCES = ("device.h", "eval_pass.hip", "kernels.hip", "launch.h", "internal.h", "api.cpp")


def source_hash():
    """sha256 of the kernel and launch sources."""
    h = hashlib.sha256()
    for f in SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2508_05370_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def _profile_value(path, key, workload, chunk):
    """A figure from a committed rocprofv3 summary of the 16M-plan workload in one call; None
    unless it was taken on this workload with the sources as they are now (hash recorded there)."""
    if workload != 3 or chunk != 0 or not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("sources_sha256") != source_hash():
        return None
    return int(kv[key])


def measured_traffic(workload, chunk):
    """HBM bytes per evaluation call, from the FETCH_SIZE/WRITE_SIZE summary."""
    return _profile_value(TRAFFIC_FILE, "traffic_bytes_per_launch", workload, chunk)


def measured_valu(workload, chunk):
    """VALU lane-ops executed per evaluation call by the evaluation kernels, from the SQ counter summary."""
    return _profile_value(SQ_FILE, "valu_lane_ops_per_launch", workload, chunk)


def timed_loop(torch, steps, fn):
    fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return time.perf_counter() - t0


def leg_same_plans(torch, B, sim, dp, out, best, n, steps, name, hdr_or):
    d = dict(dp, hdr=dp["hdr"] | hdr_or)

    def step():
        sim.eval_plans(d, out=out)
        sim.argmin(out, out=best)
    dt = timed_loop(torch, steps, step)
    bt, bi = B.best_tuple(best)
    return {"workload": name, "plans_per_s": round(n * steps / dt, 1), "steps": steps,
            "ms_per_step": round(dt / steps * 1e3, 4), "argmin": [bi, bt]}


def leg_moe(torch, B, W, steps):
    """Mixtral-8x7B-shaped MoE workload: 4M plans with EP in {1, 2, 4, 8}, one call per step."""
    w = W.workload(4)
    n = w["n_plans"]
    p = W.plans(w, 0, n)
    hashes = input_hashes(p)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    out = torch.empty(n, dtype=torch.int64, device="cuda")
    best = torch.empty(2, dtype=torch.int64, device="cuda")

    def step():
        sim.eval_plans(dp, out=out)
        sim.argmin(out, out=best)
    dt = timed_loop(torch, steps, step)
    bt, bi = B.best_tuple(best)
    valid = int(np.count_nonzero(B.times_u64(out) != MAXU))
    ep = 1 << ((p["hdr"] >> 2) & 3).astype(np.int64)
    sim.close()
    return {"workload": w["name"], "plans": n, "valid_plans": valid,
            "plans_with_ep_gt_1": int(np.count_nonzero(ep > 1)), "plans_per_s": round(n * steps / dt, 1),
            "steps": steps, "ms_per_step": round(dt / steps * 1e3, 4), "argmin": [bi, bt],
            "input_sha256": hashes}


def leg_gpt3_chunked(torch, B, W, steps, chunk=1 << 22, nstreams=2):
    """GPT-3-175B-shaped workload: 64M plans in 4M-plan chunks alternating over two streams, one
    argmin slot per chunk, one device reduction.  Resident: all 64M plans in HBM.  End to end: each
    step also generates every chunk on the host and copies it in (pinned staging, double
    buffered), so it includes generation and PCIe."""
    w = W.workload(5)
    n = w["n_plans"]
    t0 = time.time()
    p = W.plans(w, 0, n)
    gen_s = time.time() - t0
    hashes = input_hashes(p)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    out = torch.empty(n, dtype=torch.int64, device="cuda")
    chunks = [(o, min(chunk, n - o)) for o in range(0, n, chunk)]
    slots = torch.empty(2 * len(chunks), dtype=torch.int64, device="cuda")
    best = torch.empty(2, dtype=torch.int64, device="cuda")
    streams = [torch.cuda.Stream() for _ in range(nstreams)]
    main = torch.cuda.current_stream()

    def step():
        ev = main.record_event()
        for j, (o, m) in enumerate(chunks):
            st = streams[j % nstreams]
            st.wait_event(ev)
            sim.eval_plans(dp, n=m, offset=o, out=out[o:o + m], stream=st)
            sim.argmin(out[o:o + m], index_base=o, out=slots[2 * j:2 * j + 2], stream=st)
        for st in streams:
            main.wait_stream(st)
        sim.best_reduce(slots, out=best, stream=main)
    dt = timed_loop(torch, steps, step)
    bt, bi = B.best_tuple(best)
    valid = int(np.count_nonzero(B.times_u64(out) != MAXU))
    del dp, p

    # end to end: chunk generation on the host, copy in through pinned buffers, evaluation
    pinned = [{k: torch.empty(shape, dtype=dt_, pin_memory=True) for k, (shape, dt_) in
               dict(hdr=((chunk,), torch.int32), cut=((16, chunk), torch.uint8), cls=((4, chunk), torch.int32),
                    types=((4, chunk), torch.int64)).items()} for _ in range(2)]
    dev = [{k: torch.empty(v.shape, dtype=v.dtype, device="cuda") for k, v in pinned[0].items()} for _ in range(2)]
    copied = [torch.cuda.Event() for _ in range(2)]
    done = [torch.cuda.Event() for _ in range(2)]
    e2e_best = torch.empty(2, dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for j, (o, m) in enumerate(chunks):
        b = j % 2
        if j >= 2:
            done[b].synchronize()             # the evaluation that read these buffers has finished
        q = W.plans(w, o, m)
        for k in pinned[b]:
            pinned[b][k].numpy().view(q[k].dtype)[...] = q[k]
        st = streams[b]
        with torch.cuda.stream(st):
            for k in dev[b]:
                dev[b][k].copy_(pinned[b][k], non_blocking=True)
            copied[b].record(st)
            sim.eval_plans(dev[b], n=m, out=out[o:o + m], stream=st)
            sim.argmin(out[o:o + m], index_base=o, out=slots[2 * j:2 * j + 2], stream=st)
            done[b].record(st)
    for st in streams:
        main.wait_stream(st)
    sim.best_reduce(slots, out=e2e_best, stream=main)
    torch.cuda.synchronize()
    e2e = time.perf_counter() - t0
    e2e_t, e2e_i = B.best_tuple(e2e_best)
    sim.close()
    return {"workload": w["name"], "plans": n, "valid_plans": valid,
            "chunks": {"plans": chunk, "streams": nstreams}, "plans_per_s": round(n * steps / dt, 1),
            "steps": steps, "ms_per_step": round(dt / steps * 1e3, 4), "argmin": [bi, bt],
            "end_to_end_with_generation_and_pcie": {"plans_per_s": round(n / e2e, 1), "seconds": round(e2e, 3),
                                                    "argmin": [e2e_i, e2e_t]},
            "host_generation_s_for_all_plans": round(gen_s, 2), "input_sha256": hashes}


def cpu_baseline(p, got, w, one_thread_plans):
    """The oracle as it stands over every plan of the workload on the host's CPU share, and on one
    thread over a bounded prefix; mismatches against the GPU and its argmin."""
    from oracle import oracle as O
    o = O.Oracle(w["model"], w["cluster"])
    n = p["hdr"].shape[0]
    threads = host_threads()
    c0 = time.perf_counter()
    ref = o.eval(p, nthreads=threads)
    spent = time.perf_counter() - c0
    mism = int(np.count_nonzero(ref != got))
    i = int(np.argmin(ref))
    m = min(one_thread_plans, n)
    sub = {k: (v[:m] if k == "hdr" else np.ascontiguousarray(v[:, :m])) for k, v in p.items()}
    c0 = time.perf_counter()
    o.eval(sub, nthreads=1)
    one = time.perf_counter() - c0
    return {"value": round(n / spent, 1), "unit": "plans/s", "cores": threads, "kind": "oracle",
            "sample": "every plan of the workload (%d plans, %.1f s on %d threads)" % (n, spent, threads),
            "one_thread": {"plans_per_s": round(m / one, 1), "sample": "first %d plans (%.1f s)" % (m, one)},
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "parity_mismatches_vs_gpu": mism, "oracle_argmin": [i, int(ref[i])]}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=3, help="1..5 (3 = Llama-70B-shaped, 16M plans)")
    ap.add_argument("--plans", type=int, default=0, help="evaluate only the first N plans (0 = all)")
    ap.add_argument("--cpu", type=int, default=1, help="time the oracle over every plan (0 = skip)")
    ap.add_argument("--cpu-one-thread-plans", type=int, default=150_000)
    ap.add_argument("--no-timing", action="store_true", help="no HIP events inside the library")
    ap.add_argument("--chunk", type=int, default=0,
                    help="evaluate in chunks of this many plans on --streams streams, one argmin slot per chunk "
                         "reduced on the device (0 = one call over all plans)")
    ap.add_argument("--streams", type=int, default=2)
    ap.add_argument("--mem-steps", type=int, default=5,
                    help="also time the same plans with per-type device memory checked (0 = skip)")
    ap.add_argument("--overlap-steps", type=int, default=5,
                    help="also time the same plans with the gradient sync overlapped with the last backward (0 = skip)")
    ap.add_argument("--zb-steps", type=int, default=3,
                    help="also time the same plans in the zero-bubble pipeline order (0 = skip)")
    ap.add_argument("--il-steps", type=int, default=3,
                    help="also time as many interleaved-1F1B plans of the workload (0 = skip)")
    ap.add_argument("--layout-steps", type=int, default=5,
                    help="also time as many per-class-layout plans of the workload (0 = skip)")
    ap.add_argument("--moe-steps", type=int, default=5, help="also time the 4M-plan MoE workload (0 = skip)")
    ap.add_argument("--gpt3-steps", type=int, default=3,
                    help="also time the 64M-plan GPT-3-shaped workload in 4M-plan chunks on two streams (0 = skip)")
    ap.add_argument("--copy-calibrate", type=int, default=0, metavar="BYTES",
                    help="only run a device-to-device copy of BYTES (reference for HBM byte counters)")
    a = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print("bench.py evaluates on exactly one GPU: plans shard by index across GPUs with one 16-byte "
              "argmin exchange, which this benchmark does not run; use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2508_05370_amd import binding as B
    from paper_2508_05370_amd import workloads as W

    assert torch.cuda.is_available(), "no GPU"
    if a.copy_calibrate:
        src = torch.ones(a.copy_calibrate // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": a.copy_calibrate, "launches": 3}), flush=True)
        return
    w = W.workload(a.workload)
    n = a.plans or w["n_plans"]
    t0 = time.time()
    p = W.plans(w, 0, n)
    log("generated %d plans in %.1f s" % (n, time.time() - t0))
    hashes = input_hashes(p)
    sim = B.Sim(w["model"], w["cluster"])
    dp = B.device_plans(p)
    out = torch.empty(n, dtype=torch.int64, device="cuda")
    best = torch.empty(2, dtype=torch.int64, device="cuda")

    if a.chunk:
        chunks = [(o, min(a.chunk, n - o)) for o in range(0, n, a.chunk)]
        slots = torch.empty(2 * len(chunks), dtype=torch.int64, device="cuda")
        streams = [torch.cuda.Stream() for _ in range(max(1, a.streams))]
        main = torch.cuda.current_stream()

        def step():
            # chunks alternate over the streams; each writes its own argmin slot
            ev = main.record_event()
            for j, (o, m) in enumerate(chunks):
                st = streams[j % len(streams)]
                st.wait_event(ev)
                sim.eval_plans(dp, n=m, offset=o, out=out[o:o + m], stream=st)
                sim.argmin(out[o:o + m], index_base=o, out=slots[2 * j:2 * j + 2], stream=st)
            for st in streams:
                main.wait_stream(st)
            sim.best_reduce(slots, out=best, stream=main)
    else:
        def step():
            sim.eval_plans(dp, out=out)
            sim.argmin(out, out=best)

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    got = B.times_u64(out)
    valid = got != MAXU
    moe = bool(w["model"].get("experts"))
    ops = pipeline_ops(p, valid)
    setup = setup_ops(p, valid, moe)
    calls_per_step = len(range(0, n, a.chunk)) if a.chunk else 1

    [sim.get_timing(k) for k in range(4)]          # clear
    sim.get_skipped_ops()
    timed = 0 if a.no_timing else 1
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(a.steps):
        # the library's kernel events and work counters ride along on the
        # last step only: they cost about a tenth of a step's time
        if timed and i == a.steps - timed:
            sim.set_timing(True)
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    skipped = sim.get_skipped_ops() if not a.no_timing else 0
    sim.set_timing(False)
    elapsed = t1 - t0
    value = n * a.steps / elapsed
    best_t, best_i = B.best_tuple(best)

    roof = None
    extra = {}
    if not a.no_timing:
        pipe_ms, pipe_n = sim.get_timing(0)
        setup_ms, setup_n = sim.get_timing(1)
        call_ms, call_n = sim.get_timing(2)
        defer_ms, defer_n = sim.get_timing(3)
        node_rate = B.measure_node_rate()
        peak = min(PEAK_VALU_SPEC, 3 * node_rate)
        # one launch = one sim_eval_plans call (all its kernels, on all its
        # streams), timed by the library's events on the call's stream
        avg_ms = call_ms / max(call_n, 1)
        full_per_launch = float(ops.sum()) / calls_per_step
        int32_per_launch = float(pipeline_ops(p, valid, 7, 2).sum()) / calls_per_step
        rec_per_launch = full_per_launch - skipped / timed / calls_per_step
        setup_per_launch = float(setup.sum()) / calls_per_step
        work = rec_per_launch + setup_per_launch
        achieved = work / (avg_ms * 1e-3)
        roof = {"bound": "alu", "achieved": round(achieved / 1e12, 3), "peak": round(peak / 1e12, 3),
                "unit": "TOP/s", "frac": round(achieved / peak, 4),
                "traffic": None if a.plans else measured_traffic(a.workload, a.chunk),
                "kernel": "one sim_eval_plans call: k_fill32, k_prep, k_scan, k_scatter, k_eval x4 groups, "
                          "k_variant x4, k_defer_hist, k_defer_sort, k_deferred, k_redo_u64 per 2M-plan chunk",
                "avg_launch_ms": round(avg_ms, 4), "launches": call_n,
                "work_per_launch": work,
                "recurrence_ops_per_launch": rec_per_launch, "setup_ops_per_launch": setup_per_launch,
                "full_recurrence_ops_per_launch": full_per_launch,
                "skipped_by_periodic_shortcut": round(1 - rec_per_launch / full_per_launch, 4),
                "peak_spec": round(PEAK_VALU_SPEC / 1e12, 3),
                "peak_measured_node_probe": round(3 * node_rate / 1e12, 3),
                "node_probe_nodes_per_s": round(node_rate, 1),
                # labelled comparisons, not the roofline fraction: the int32 count of every node (7 ops with a
                # cross-stage input, 2 without) whether the shortcut skips it or not, over the call
                "int32_all_nodes_ops_per_launch": int32_per_launch,
                "int32_all_nodes_rate_over_peak": round(int32_per_launch / (avg_ms * 1e-3) / peak, 4)}
        # every VALU instruction the evaluation kernels execute (setup, recurrence, syncs), from counters
        valu = None if a.plans else measured_valu(a.workload, a.chunk)
        roof["valu_lane_ops_per_launch_counters"] = valu
        roof["valu_issue_frac_counters"] = None if valu is None else round(valu / (avg_ms * 1e-3) / PEAK_VALU_SPEC, 4)
        extra = {"timed_steps_with_kernel_events": timed,
                 "prep_ms_per_step": round(setup_ms / timed, 4),
                 "first_pass_span_ms_per_step": round(pipe_ms / timed, 4),
                 "deferred_pass_ms_per_step": round(defer_ms / timed, 4),
                 "eval_call_ms_per_step": round(call_ms / timed, 4)}

    # The same sweep with device memory capacities: plans that do not fit become invalid
    mem = None
    if a.mem_steps > 0 and not a.chunk:
        wm = W.with_memory(w)
        simm = B.Sim(wm["model"], wm["cluster"])

        def mstep():
            simm.eval_plans(dp, out=out)
            simm.argmin(out, out=best)
        dt = timed_loop(torch, a.mem_steps, mstep)
        fit = int(np.count_nonzero(B.times_u64(out) != MAXU))
        mb_t, mb_i = B.best_tuple(best)
        mem = {"workload": wm["name"], "memory_GiB": [t["mem_bytes"] >> 30 for t in wm["cluster"]["types"]],
               "plans_per_s": round(n * a.mem_steps / dt, 1), "steps": a.mem_steps,
               "ms_per_step": round(dt / a.mem_steps * 1e3, 4), "feasible_plans": fit, "argmin": [mb_i, mb_t]}
        simm.close()

    ovl = None
    if a.overlap_steps > 0 and not a.chunk:
        ovl = leg_same_plans(torch, B, sim, dp, out, best, n, a.overlap_steps, w["name"] + "/overlap", 1 << 13)
    zb = None
    if a.zb_steps > 0 and not a.chunk:
        zb = leg_same_plans(torch, B, sim, dp, out, best, n, a.zb_steps, w["name"] + "/zero-bubble", 1 << 16)

    # Plans with a per-class layout (each replica class its own TP degree, depth and layer split)
    lay = None
    if a.layout_steps > 0 and not a.chunk:
        t0 = time.time()
        ph = W.het_plans(w, 0, n)
        log("generated %d per-class-layout plans in %.1f s" % (n, time.time() - t0))
        dh = B.device_plans(ph)
        del ph

        def hstep():
            sim.eval_plans(dh, out=out)
            sim.argmin(out, out=best)
        dt = timed_loop(torch, a.layout_steps, hstep)
        hb_t, hb_i = B.best_tuple(best)
        lay = {"workload": w["name"] + "/per-class-layout", "plans_per_s": round(n * a.layout_steps / dt, 1),
               "steps": a.layout_steps, "ms_per_step": round(dt / a.layout_steps * 1e3, 4),
               "valid_plans": int(np.count_nonzero(B.times_u64(out) != MAXU)), "argmin": [hb_i, hb_t]}
        del dh

    # Interleaved 1F1B plans (v model chunks per device) of the same workload
    il = None
    if a.il_steps > 0 and not a.chunk:
        t0 = time.time()
        pi = W.interleaved_plans(w, 0, n)
        log("generated %d interleaved plans in %.1f s" % (n, time.time() - t0))
        di = B.device_plans(pi)

        def istep():
            sim.eval_plans(di, out=out)
            sim.argmin(out, out=best)
        dt = timed_loop(torch, a.il_steps, istep)
        ib_t, ib_i = B.best_tuple(best)
        ivalid = B.times_u64(out) != MAXU
        v = (((pi["hdr"] >> 14) & 3) + 1).astype(np.int64)
        # schedule nodes: every device runs 2 M v ops per class
        nodes = pipeline_ops(pi, ivalid, per_node=1, first=1) * v
        il = {"workload": w["name"] + "/interleaved", "plans_per_s": round(n * a.il_steps / dt, 1),
              "steps": a.il_steps, "ms_per_step": round(dt / a.il_steps * 1e3, 4),
              "valid_plans": int(ivalid.sum()), "argmin": [ib_i, ib_t],
              "schedule_nodes_per_s": round(float(nodes.sum()) * a.il_steps / dt, 1)}
        del di, pi
    del dp
    sim.close()

    moe_leg = leg_moe(torch, B, W, a.moe_steps) if a.moe_steps > 0 else None
    gpt3_leg = leg_gpt3_chunked(torch, B, W, a.gpt3_steps) if a.gpt3_steps > 0 else None

    # CPU baseline: the oracle as it stands, over every plan of the same workload
    cpu = cpu_baseline(p, got, w, a.cpu_one_thread_plans) if a.cpu else None
    if cpu is not None:
        cpu["argmin_matches_gpu"] = cpu["oracle_argmin"] == [best_i, best_t]

    rec = {"metric": METRIC, "value": round(value, 1), "unit": "plans/s", "n_gpus": 1, "steps": a.steps,
           "warmup": a.warmup, "ms_per_step": round(elapsed / a.steps * 1e3, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
           "config": {"workload": w["name"], "plans": n, "valid_plans": int(valid.sum()),
                      "chunks": ({"plans": a.chunk, "streams": a.streams} if a.chunk else None),
                      "argmin": [best_i, best_t], "mean_pipeline_ops_per_plan": round(float(ops.mean()), 1),
                      "mean_setup_ops_per_plan": round(float(setup.mean()), 1), "input_sha256": hashes},
           "roofline": roof, "cpu_baseline": cpu}
    rec.update(extra)
    rec["memory_check"] = mem
    rec["dp_overlap"] = ovl
    rec["per_class_layout"] = lay
    rec["interleaved"] = il
    rec["zero_bubble"] = zb
    rec["moe_workload"] = moe_leg
    rec["gpt3_workload_chunked"] = gpt3_leg
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
