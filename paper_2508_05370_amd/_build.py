"""Build the HIP library (libhetsim.so, gfx950) and the input generator in-tree."""
import concurrent.futures
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libhetsim.so")

ARCH = "gfx950"
HIP_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
             # packed fp32 VALU forms are kept out of every kernel
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# the pipeline recurrence carries integer times in fp64: no NaN/inf ever occurs,
# which lets max() compile to one v_max_f64 (no reassociation is enabled)
KERNEL_FLAGS = ["-ffinite-math-only"]
# (source, object, extra flags): the common kernels, the C ABI, the table
# builder, and one object per evaluation-pass variant -- table mode (0..2) x
# plan layout (shared, per class) x pass (first, deferred), and the variant
# pass (overlap and zero-bubble pipelines, shared layout) per table mode --
# so that they compile in parallel
SOURCES = [("kernels.hip", "kernels.o", KERNEL_FLAGS), ("api.cpp", "api.o", []), ("tables.cpp", "tables.o", [])]
SOURCES += [("eval_pass.hip", "eval_pass_m%d_h%d_p%d.o" % (m, h, p),
             KERNEL_FLAGS + ["-DHETSIM_MODE=%d" % m, "-DHETSIM_HET=%d" % h, "-DHETSIM_PASS=%d" % p])
            for p in (1, 0) for m in range(3) for h in range(2)]
SOURCES += [("eval_pass.hip", "eval_pass_m%d_h0_p2.o" % m,
             KERNEL_FLAGS + ["-DHETSIM_MODE=%d" % m, "-DHETSIM_HET=0", "-DHETSIM_PASS=2"]) for m in range(3)]


def _jobs():
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:
        return max(1, os.cpu_count() or 1)


def _compile(cmd):
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    text = "\n".join(ln for ln in proc.stdout.decode(errors="replace").splitlines() if "packed-fp32-ops" not in ln)
    return proc.returncode, text


def _stale(src, obj):
    """An object is stale when older than its source or any header of the library."""
    if not os.path.exists(obj):
        return True
    deps = [src] + [os.path.join(d, f) for d in (CSRC, INCLUDE) for f in os.listdir(d) if f.endswith(".h")]
    return os.path.getmtime(obj) < max(os.path.getmtime(x) for x in deps)


def build(force=True, verbose=False, incremental=False):
    """Compile every object and link the library.  incremental: recompile only stale objects."""
    if not force and not incremental and os.path.exists(LIB):
        return LIB
    os.makedirs(BUILD, exist_ok=True)
    cmds = [["hipcc", *HIP_FLAGS, *extra, "-I", INCLUDE, "-c", os.path.join(CSRC, src), "-o", os.path.join(BUILD, obj)]
            for src, obj, extra in SOURCES
            if not incremental or _stale(os.path.join(CSRC, src), os.path.join(BUILD, obj))]
    with concurrent.futures.ThreadPoolExecutor(max_workers=_jobs()) as pool:
        results = list(pool.map(_compile, cmds))
    for cmd, (rc, text) in zip(cmds, results):
        if rc != 0:
            raise RuntimeError("hipcc failed: %s\n%s" % (" ".join(cmd), text))
        if verbose and text.strip():
            print(text)
    objs = [os.path.join(BUILD, obj) for _, obj, _ in SOURCES]
    tmp = LIB + ".tmp"
    subprocess.run(["hipcc", "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, "-o", tmp], check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    import sys
    print(build(verbose=True, incremental="--incremental" in sys.argv))
