"""The oracle built with AddressSanitizer + UndefinedBehaviorSanitizer, and with ThreadSanitizer.

CPU only.  oracle.c is compiled twice more into a temporary directory: once with
-fsanitize=address,undefined (no recovery: the first report aborts), once with -fsanitize=thread.
A child Python process preloads the matching sanitizer runtime, loads the instrumented build
(the wrapper takes the library named by HETSIM_ORACLE_LIB) and evaluates plans of every kind --
shared layout, overlap, zero-bubble, interleaved, per-class layout -- on the five workloads and on
random configurations with cluster options and device memory, on four threads, plus the stage
records and the per-device memory of some of them.  The child must exit cleanly (a sanitizer
report fails it) and its times must equal the plain build's.
"""
import os
import subprocess
import sys
import tempfile

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
N = 240


def cases(workloads):
    """(name, model, cluster, plans) for every plan kind on the five workloads and four random
    configurations (cluster options on, device memory on for some)."""
    from test_gpu_random_configs import OPTIONS, _config
    out = []

    def kinds(tag, m, c, s0):
        p = workloads.random_plans(m, c, s0, 0, N)
        out.append((tag + "/plain", m, c, p))
        for kind, bit in (("overlap", 13), ("zero-bubble", 16)):
            q = {k: v.copy() for k, v in p.items()}
            q["hdr"] |= np.uint32(1 << bit)
            out.append((tag + "/" + kind, m, c, q))
        out.append((tag + "/interleaved", m, c, workloads.random_plans_il(m, c, s0 + 1, 0, N)))
        out.append((tag + "/per-class", m, c, workloads.random_plans_het(m, c, s0 + 2, 0, N)))

    w1 = workloads.workload(1)
    out.append(("workload1/exhaustive", w1["model"], w1["cluster"], workloads.plans(w1, 0, N)))
    for idx in (2, 3, 4, 5):
        w = workloads.workload(idx)
        kinds("workload%d" % idx, w["model"], w["cluster"], 0x5A170000 + idx)
        wm = workloads.with_memory(w)
        out.append(("workload%d/memory" % idx, wm["model"], wm["cluster"], workloads.plans(wm, 0, N)))
    for seed in (1, 5, 9, 13):
        _, m, c, s0 = _config(workloads, seed)
        c = dict(c, **{k: True for k in OPTIONS})
        kinds("random%d" % seed, m, c, s0)
    return out


def child(out_path):
    """Runs in the instrumented process: evaluate every case, save the times."""
    from oracle import oracle as O
    from paper_2508_05370_amd import workloads as W
    res = {}
    for name, m, c, p in cases(W):
        o = O.Oracle(m, c)
        res[name] = o.eval(p, nthreads=4)
        if name.endswith("/plain") or name.endswith("/per-class"):
            for i in range(0, N, 37):
                o.detail(p, i)
                o.stage_mem(p, i)
    np.savez(out_path, **{k.replace("/", "__"): v for k, v in res.items()})


def _build(flags, path):
    subprocess.run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-std=c11", "-fPIC", "-shared", "-pthread",
                    *flags, SRC, "-o", path], check=True)


@pytest.mark.parametrize("kind", ["address,undefined", "thread"])
def test_oracle_under_sanitizers(oracle_mod, workloads, kind):
    runtime = {"address,undefined": "libasan.so", "thread": "libtsan.so"}[kind]
    rt = subprocess.run(["gcc", "-print-file-name=" + runtime], stdout=subprocess.PIPE, check=True).stdout.decode().strip()
    if not os.path.isabs(rt) or not os.path.exists(rt):
        pytest.skip("no %s runtime for gcc" % runtime)
    flags = ["-fsanitize=" + kind]
    if kind != "thread":
        flags.append("-fno-sanitize-recover=all")
    with tempfile.TemporaryDirectory() as d:
        lib = os.path.join(d, "liboracle_san.so")
        _build(flags, lib)
        out = os.path.join(d, "times.npz")
        env = dict(os.environ, HETSIM_ORACLE_LIB=lib, LD_PRELOAD=rt,
                   ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
                   UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
                   TSAN_OPTIONS="halt_on_error=1:report_signal_unsafe=0")
        code = ("import sys; sys.path[:0] = [%r, %r]; import test_oracle_sanitizers as T; T.child(%r)"
                % (ROOT, os.path.join(ROOT, "tests"), out))
        proc = subprocess.run([sys.executable, "-c", code], env=env, stdout=subprocess.PIPE,
                              stderr=subprocess.STDOUT, timeout=900)
        text = proc.stdout.decode(errors="replace")
        assert proc.returncode == 0, "sanitizer run failed (%d):\n%s" % (proc.returncode, text[-4000:])
        assert "Sanitizer" not in text, text[-4000:]
        got = np.load(out)
        for name, m, c, p in cases(workloads):
            want = oracle_mod.Oracle(m, c).eval(p)
            assert np.array_equal(got[name.replace("/", "__")], want), name
