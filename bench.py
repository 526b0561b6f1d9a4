"""Throughput of batched plan evaluation on one MI355X.

One step = the whole hot path over every plan of the workload: decode and
validate, place, stage costs, bottleneck links, collectives, the 1F1B pipeline
of every replica class, the DP sync, and the argmin over all plans.  Plans are
resident in HBM before timing starts.

Prints one JSON line.  Roofline: the evaluation is bound by VALU issue.  The
1F1B recurrence costs 3 VALU ops (add, max, add) per dependent schedule node
and 1 per node without a cross-stage input, i.e. sum over classes of
M * (6 (S - 1) + 2) per plan; the library skips the steady iterations that
follow a periodic one (counted on the device while timing is on), and the
algorithmic work reported is the recurrence work that remains, per
sim_eval_plans call, over the call's duration.  The peak is 256 CUs x 64
lanes x 2.4 GHz.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_VALU = 256 * 64 * 2.4e9          # lane-ops per second (fp64 add/max issue at full rate)
METRIC = "candidate plans evaluated/sec on 1 MI355X; % of binding roofline"
MAXU = np.uint64(2**64 - 1)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def pipeline_ops(p, valid, per_node=3, first=1):
    """VALU ops of the whole pipeline recurrence, per plan: `per_node` per schedule node with a
    cross-stage input, `first` per node without one (3 and 1 in fp64 as the kernels run it; the
    int32 count of the same nodes is 7 and 2)."""
    hdr = p["hdr"]
    S = (((hdr >> 4) & 15) + 1).astype(np.int64)
    G = ((hdr >> 8) & 3) + 1
    ops = np.zeros(hdr.shape[0], dtype=np.int64)
    for c in range(4):
        reps = (p["cls"][c] & 0xFFFF).astype(np.int64)
        nmb = (p["cls"][c] >> 16).astype(np.int64)
        has = (G > c) & valid & (reps > 0)
        M = np.where(has, -(-nmb // np.maximum(reps, 1)), 0)
        ops += 2 * M * (per_node * (S - 1) + first)
    return ops


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "eval_llama70b_16M_hbm_traffic.txt")
SQ_FILE = os.path.join(ROOT, "profiles", "eval_llama70b_16M_sq_counters.txt")


def source_hash():
    """sha256 of the kernel and launch sources (kernels.hip, then api.cpp)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("kernels.hip", "api.cpp"):
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=3, help="1..5 (3 = Llama-70B-shaped, 16M plans)")
    ap.add_argument("--plans", type=int, default=0, help="evaluate only the first N plans (0 = all)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="oracle time budget for the CPU baseline")
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
    ap.add_argument("--copy-calibrate", type=int, default=0, metavar="BYTES",
                    help="only run a device-to-device copy of BYTES (reference for HBM byte counters)")
    a = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print("bench.py evaluates on exactly one GPU: plans shard by index across GPUs with one 16-byte "
              "argmin exchange, which this build does not run; use --gpus 1", file=sys.stderr)
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
    ops = pipeline_ops(p, valid)
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
        # one launch = one sim_eval_plans call (all its kernels, on all its
        # streams), timed by the library's events on the call's stream
        avg_ms = call_ms / max(call_n, 1)
        full_per_launch = float(ops.sum()) / calls_per_step
        int32_per_launch = float(pipeline_ops(p, valid, 7, 2).sum()) / calls_per_step
        ops_per_launch = full_per_launch - skipped / timed / calls_per_step
        achieved = ops_per_launch / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "alu", "achieved": round(achieved, 3), "peak": round(PEAK_VALU / 1e12, 3),
                "unit": "TOP/s", "frac": round(achieved * 1e12 / PEAK_VALU, 4),
                "traffic": None if a.plans else measured_traffic(a.workload, a.chunk),
                "kernel": "sim_eval_plans call: k_prep, k_scan, k_scatter, k_eval x4 groups, k_deferred, "
                          "k_redo_u64 per 2M-plan chunk",
                "avg_launch_ms": round(avg_ms, 4), "launches": call_n, "ops_per_launch": ops_per_launch,
                "full_recurrence_ops_per_launch": full_per_launch,
                "skipped_by_periodic_shortcut": round(1 - ops_per_launch / full_per_launch, 4),
                # the int32 count of every node (7 ops with a cross-stage input, 2 without), shortcut or
                # not: what the evaluation would cost without the shortcut, in 32-bit integer ops
                "int32_all_nodes_ops_per_launch": int32_per_launch,
                "int32_all_nodes_rate_frac": round(int32_per_launch / (avg_ms * 1e-3) / PEAK_VALU, 4)}
        # every VALU instruction the evaluation kernels execute (setup, recurrence, syncs), from counters
        valu = None if a.plans else measured_valu(a.workload, a.chunk)
        roof["valu_lane_ops_per_launch_counters"] = valu
        roof["valu_issue_frac"] = None if valu is None else round(valu / (avg_ms * 1e-3) / PEAK_VALU, 4)
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
        simm.eval_plans(dp, out=out)
        simm.argmin(out, out=best)
        torch.cuda.synchronize()
        m0 = time.perf_counter()
        for _ in range(a.mem_steps):
            simm.eval_plans(dp, out=out)
            simm.argmin(out, out=best)
        torch.cuda.synchronize()
        m1 = time.perf_counter()
        fit = int(np.count_nonzero(B.times_u64(out) != MAXU))
        mb_t, mb_i = B.best_tuple(best)
        mem = {"workload": wm["name"], "memory_GiB": [t["mem_bytes"] >> 30 for t in wm["cluster"]["types"]],
               "plans_per_s": round(n * a.mem_steps / (m1 - m0), 1), "steps": a.mem_steps,
               "ms_per_step": round((m1 - m0) / a.mem_steps * 1e3, 4), "feasible_plans": fit,
               "argmin": [mb_i, mb_t]}
        simm.close()

    # The same plans with the gradient sync overlapped with each stage's last backward pass
    ovl = None
    if a.overlap_steps > 0 and not a.chunk:
        dov = dict(dp, hdr=dp["hdr"] | (1 << 13))
        sim.eval_plans(dov, out=out)
        sim.argmin(out, out=best)
        torch.cuda.synchronize()
        o0 = time.perf_counter()
        for _ in range(a.overlap_steps):
            sim.eval_plans(dov, out=out)
            sim.argmin(out, out=best)
        torch.cuda.synchronize()
        o1 = time.perf_counter()
        ob_t, ob_i = B.best_tuple(best)
        ovl = {"workload": w["name"] + "/overlap", "plans_per_s": round(n * a.overlap_steps / (o1 - o0), 1),
               "steps": a.overlap_steps, "ms_per_step": round((o1 - o0) / a.overlap_steps * 1e3, 4),
               "argmin": [ob_i, ob_t]}
        del dov

    # Plans with a per-class layout (each replica class its own TP degree, depth and layer split)
    lay = None
    if a.layout_steps > 0 and not a.chunk:
        t0 = time.time()
        ph = W.het_plans(w, 0, n)
        log("generated %d per-class-layout plans in %.1f s" % (n, time.time() - t0))
        dh = B.device_plans(ph)
        del ph
        sim.eval_plans(dh, out=out)
        sim.argmin(out, out=best)
        torch.cuda.synchronize()
        h0 = time.perf_counter()
        for _ in range(a.layout_steps):
            sim.eval_plans(dh, out=out)
            sim.argmin(out, out=best)
        torch.cuda.synchronize()
        h1 = time.perf_counter()
        hb_t, hb_i = B.best_tuple(best)
        lay = {"workload": w["name"] + "/per-class-layout", "plans_per_s": round(n * a.layout_steps / (h1 - h0), 1),
               "steps": a.layout_steps, "ms_per_step": round((h1 - h0) / a.layout_steps * 1e3, 4),
               "valid_plans": int(np.count_nonzero(B.times_u64(out) != MAXU)), "argmin": [hb_i, hb_t]}
        del dh

    # The same plans in the zero-bubble order (backward split into input and weight gradients)
    zb = None
    if a.zb_steps > 0 and not a.chunk:
        dz = dict(dp, hdr=dp["hdr"] | (1 << 16))
        sim.eval_plans(dz, out=out)
        sim.argmin(out, out=best)
        torch.cuda.synchronize()
        z0 = time.perf_counter()
        for _ in range(a.zb_steps):
            sim.eval_plans(dz, out=out)
            sim.argmin(out, out=best)
        torch.cuda.synchronize()
        z1 = time.perf_counter()
        zb_t, zb_i = B.best_tuple(best)
        zb = {"workload": w["name"] + "/zero-bubble", "plans_per_s": round(n * a.zb_steps / (z1 - z0), 1),
              "steps": a.zb_steps, "ms_per_step": round((z1 - z0) / a.zb_steps * 1e3, 4),
              "argmin": [zb_i, zb_t]}
        del dz

    # Interleaved 1F1B plans (v model chunks per device) of the same workload
    il = None
    if a.il_steps > 0 and not a.chunk:
        t0 = time.time()
        pi = W.interleaved_plans(w, 0, n)
        log("generated %d interleaved plans in %.1f s" % (n, time.time() - t0))
        di = B.device_plans(pi)
        sim.eval_plans(di, out=out)
        sim.argmin(out, out=best)
        torch.cuda.synchronize()
        i0 = time.perf_counter()
        for _ in range(a.il_steps):
            sim.eval_plans(di, out=out)
            sim.argmin(out, out=best)
        torch.cuda.synchronize()
        i1 = time.perf_counter()
        ib_t, ib_i = B.best_tuple(best)
        ivalid = B.times_u64(out) != MAXU
        v = (((pi["hdr"] >> 14) & 3) + 1).astype(np.int64)
        # schedule nodes: every device runs 2 M v ops per class
        nodes = pipeline_ops(pi, ivalid, per_node=1, first=1) * v
        il = {"workload": w["name"] + "/interleaved", "plans_per_s": round(n * a.il_steps / (i1 - i0), 1),
              "steps": a.il_steps, "ms_per_step": round((i1 - i0) / a.il_steps * 1e3, 4),
              "valid_plans": int(ivalid.sum()), "argmin": [ib_i, ib_t],
              "schedule_nodes_per_s": round(float(nodes.sum()) * a.il_steps / (i1 - i0), 1)}
        del di, pi

    # CPU baseline: the oracle as it stands, on a bounded prefix of the same plans
    cpu = None
    if a.cpu_seconds > 0:
        from oracle import oracle as O
        o = O.Oracle(w["model"], w["cluster"])
        threads = min(16, os.cpu_count() or 1)
        done, spent, mism, blk = 0, 0.0, 0, 100_000
        while spent < a.cpu_seconds and done < n:
            m = min(blk, n - done)
            sub = {k: (v[done:done + m] if k == "hdr" else np.ascontiguousarray(v[:, done:done + m]))
                   for k, v in p.items()}
            c0 = time.perf_counter()
            ref = o.eval(sub, nthreads=threads)
            spent += time.perf_counter() - c0
            mism += int(np.count_nonzero(ref != got[done:done + m]))
            done += m
        cpu = {"value": round(done / spent, 1), "unit": "plans/s", "cores": threads, "kind": "oracle",
               "sample": "first %d plans of the workload (%.1f s)" % (done, spent),
               "parity_mismatches_vs_gpu": mism}

    rec = {"metric": METRIC, "value": round(value, 1), "unit": "plans/s", "n_gpus": 1, "steps": a.steps,
           "warmup": a.warmup, "ms_per_step": round(elapsed / a.steps * 1e3, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
           "config": {"workload": w["name"], "plans": n, "valid_plans": int(valid.sum()),
                      "chunks": ({"plans": a.chunk, "streams": a.streams} if a.chunk else None),
                      "argmin": [best_i, best_t], "mean_pipeline_ops_per_plan": round(float(ops.mean()), 1)},
           "roofline": roof, "cpu_baseline": cpu}
    rec.update(extra)
    rec["memory_check"] = mem
    rec["dp_overlap"] = ovl
    rec["per_class_layout"] = lay
    rec["interleaved"] = il
    rec["zero_bubble"] = zb
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
