"""The C-ABI library: loads, exports every declared entry point, and validates
descriptors on the host (no GPU needed for any of these)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def B():
    from paper_2508_05370_amd import binding
    return binding


def _declared():
    src = open(os.path.join(ROOT, "include", "hetsim.h")).read()
    return sorted(set(re.findall(r"^\s*(?:int|void|const char\*)\s+(sim_\w+)\s*\(", src, re.M)))


def test_exports_every_declared_symbol(B):
    L = B.lib()
    names = _declared()
    assert set(names) == set(B.EXPORTS)
    for n in names:
        assert hasattr(L, n), n


def test_strerror(B):
    L = B.lib()
    for code in (0, -1, -2, -3, -4, -5):
        assert L.sim_strerror(code)
    assert b"allocation-free" in L.sim_strerror(B.SIM_ESIZE)
    assert L.sim_strerror(-99) == b"unknown error"


def _create(B, m, c):
    md, k1 = B.model_desc(m)
    cd, k2 = B.cluster_desc(c)
    h = C.c_void_p()
    rc = B.lib().sim_create(C.byref(md), C.byref(cd), C.byref(h))
    return rc, h


@pytest.mark.parametrize("field,value", [
    ("L", 0), ("L", 256), ("heads", 7), ("kv_heads", 5), ("seq", 0), ("dtype_bytes", 0), ("mbs", []),
    ("mbs", [1, 2, 3, 4, 5]), ("mbs", [0]), ("gated", 2), ("ffn", 0), ("opt_bytes", 65)])
def test_create_rejects_bad_model(B, workloads, field, value):
    w = workloads.workload(1)
    m = dict(w["model"])
    m[field] = value
    if field == "mbs" and len(value) > 4:
        with pytest.raises(IndexError):
            B.model_desc(m)
        return
    rc, h = _create(B, m, w["cluster"])
    assert rc == B.SIM_EINVAL and not h.value


@pytest.mark.parametrize("field,value", [
    ("dev_per_node", 3), ("dev_per_node", 128), ("tflops", 0), ("hbm_GBps", 0), ("nic_MBps", 0),
    ("nic_MBps", 15), ("intra_MBps", 0), ("pcie_MBps", 8), ("n_nodes", 0), ("intra_alpha_ps", 2**41)])
def test_create_rejects_bad_cluster(B, workloads, field, value):
    w = workloads.workload(1)
    c = {**w["cluster"], "types": [dict(t) for t in w["cluster"]["types"]]}
    c["types"][1][field] = value
    rc, h = _create(B, w["model"], c)
    assert rc == B.SIM_EINVAL and not h.value


def test_create_rejects_zero_device_memory(B, workloads):
    """Device memory is optional for the whole cluster, but a given capacity must be >= 1 byte."""
    w = workloads.with_memory(workloads.workload(1), [40, 80])
    w["cluster"]["types"][1]["mem_bytes"] = 0
    rc, h = _create(B, w["model"], w["cluster"])
    assert rc == B.SIM_EINVAL and not h.value


def test_create_rejects_bad_moe_loads(B, workloads):
    w = workloads.workload(4)
    m = dict(w["model"])
    q = np.array(m["load_q16"])
    q[3, 0] += 1                                 # a row no longer sums to 2^16
    m["load_q16"] = q
    rc, _ = _create(B, m, w["cluster"])
    assert rc == B.SIM_EINVAL
    m["load_q16"] = None
    rc, _ = _create(B, m, w["cluster"])
    assert rc == B.SIM_EINVAL


def test_create_rejects_overflowing_descriptor(B, workloads):
    w = workloads.workload(5)
    m = dict(w["model"], global_batch=2**31 - 1)
    c = {**w["cluster"], "types": [dict(t) for t in w["cluster"]["types"]]}
    for t in c["types"]:
        t["tflops"] = 1
    rc, _ = _create(B, m, c)
    assert rc == B.SIM_ERANGE


def test_null_arguments(B):
    L = B.lib()
    assert L.sim_create(None, None, None) == B.SIM_EINVAL
    assert L.sim_eval_plans(None, None, 0, None, None) == B.SIM_EINVAL
    assert L.sim_eval_plans_noalloc(None, None, 0, None, None) == B.SIM_EINVAL
    assert L.sim_eval_stages(None, None, 0, None, None, None) == B.SIM_EINVAL
    assert L.sim_eval_memory(None, None, 0, None, None) == B.SIM_EINVAL
    assert L.sim_argmin(None, None, 0, 0, None, None) == B.SIM_EINVAL
    assert L.sim_best_reduce(None, None, 0, None, None) == B.SIM_EINVAL
    assert L.sim_set_timing(None, 1) == B.SIM_EINVAL
    L.sim_destroy(None)


def test_binding_structs_match_the_header(B, tmp_path):
    """Every descriptor the binding passes has the header's layout: each field's offset and each
    struct's size, as the C compiler lays them out, equal the ctypes mirror's."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = {"sim_model_desc": B.ModelDesc, "sim_cluster_desc": B.ClusterDesc, "sim_plans": B.Plans,
               "sim_best": B.Best}
    lines = ["#include <stddef.h>", "#include <stdio.h>", '#include "hetsim.h"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append('  printf("%s size %%zu\\n", sizeof(%s));' % (cname, cname))
        for f, _ in py._fields_:
            lines.append('  printf("%s %s %%zu\\n", offsetof(%s, %s));' % (cname, f, cname, f))
    lines += ["  return 0;", "}"]
    src = tmp_path / "probe.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "probe"
    subprocess.run([cc, "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {tuple(x.split()[:2]): int(x.split()[2]) for x in out if x}
    for cname, py in structs.items():
        assert got[(cname, "size")] == C.sizeof(py), cname
        for f, _ in py._fields_:
            assert got[(cname, f)] == getattr(py, f).offset, (cname, f)
