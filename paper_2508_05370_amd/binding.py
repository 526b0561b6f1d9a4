"""Thin ctypes binding of libhetsim.so (include/hetsim.h).

Argument marshalling only: descriptors are packed into the C structs, torch
tensors provide device memory and the current HIP stream.  Every step of the
evaluation runs in the library's HIP kernels; there is no host fallback, and a
missing library raises.
"""
import ctypes as C
import os

import numpy as np

from . import _build

SIM_OK, SIM_EINVAL, SIM_ERANGE, SIM_ENOMEM, SIM_EHIP, SIM_ESIZE = 0, -1, -2, -3, -4, -5
SIM_NOALLOC_MAX_PLANS, SIM_NOALLOC_MAX_PLANS_PER_CLASS = 1 << 18, 1 << 16
TIME_INVALID = 2**64 - 1

_lib = None


class ModelDesc(C.Structure):
    _fields_ = [("n_layers", C.c_uint32), ("hidden", C.c_uint32), ("heads", C.c_uint32), ("kv_heads", C.c_uint32),
                ("ffn", C.c_uint32), ("gated", C.c_uint32), ("vocab", C.c_uint32), ("learned_pos", C.c_uint32),
                ("seq", C.c_uint32), ("dtype_bytes", C.c_uint32), ("global_batch", C.c_uint32),
                ("n_mbs", C.c_uint32), ("mbs", C.c_uint32 * 4), ("grad_bytes", C.c_uint32),
                ("param_bytes", C.c_uint32), ("experts", C.c_uint32), ("topk", C.c_uint32),
                ("expert_ffn", C.c_uint32), ("load_q16", C.c_void_p), ("opt_bytes", C.c_uint32)]


class ClusterDesc(C.Structure):
    _fields_ = [("n_types", C.c_uint32)] + [(k, C.c_void_p) for k in (
        "n_nodes", "dev_per_node", "tflops", "hbm_GBps", "intra_MBps", "pcie_MBps", "nic_MBps", "intra_alpha_ps",
        "pcie_alpha_ps", "nic_alpha_ps", "nic_MBps_dev", "intra_MBps_node", "mem_bytes")] + [
        ("rail_only", C.c_uint32), ("ccl_tree", C.c_uint32), ("contention", C.c_uint32), ("ccl_hier", C.c_uint32)]


class Plans(C.Structure):
    _fields_ = [("hdr", C.c_void_p), ("cut", C.c_void_p), ("cls", C.c_void_p), ("types", C.c_void_p),
                ("stride", C.c_int64), ("chdr", C.c_void_p), ("ccut", C.c_void_p)]


class Best(C.Structure):
    _fields_ = [("time_ps", C.c_uint64), ("index", C.c_int64)]


EXPORTS = ("sim_create", "sim_eval_plans", "sim_eval_plans_noalloc", "sim_eval_stages", "sim_eval_memory", "sim_argmin", "sim_best_reduce", "sim_set_timing",
           "sim_get_timing", "sim_get_skipped_ops", "sim_destroy", "sim_strerror", "sim_measure_node_rate")


def lib():
    """Load libhetsim.so (built in-tree; HETSIM_LIB may name another build of it)."""
    global _lib
    if _lib is None:
        path = os.environ.get("HETSIM_LIB") or _build.LIB
        if path == _build.LIB and not os.path.exists(path):
            _build.build(force=False)
        L = C.CDLL(path)
        P, I64 = C.c_void_p, C.c_int64
        L.sim_create.argtypes = [C.POINTER(ModelDesc), C.POINTER(ClusterDesc), C.POINTER(P)]
        L.sim_create.restype = C.c_int
        L.sim_eval_plans.argtypes = [P, C.POINTER(Plans), I64, P, P]
        L.sim_eval_plans.restype = C.c_int
        L.sim_eval_plans_noalloc.argtypes = [P, C.POINTER(Plans), I64, P, P]
        L.sim_eval_plans_noalloc.restype = C.c_int
        L.sim_measure_node_rate.argtypes = [C.POINTER(C.c_double), P]
        L.sim_measure_node_rate.restype = C.c_int
        L.sim_eval_stages.argtypes = [P, C.POINTER(Plans), I64, P, P, P]
        L.sim_eval_stages.restype = C.c_int
        L.sim_eval_memory.argtypes = [P, C.POINTER(Plans), I64, P, P]
        L.sim_eval_memory.restype = C.c_int
        L.sim_argmin.argtypes = [P, P, I64, I64, P, P]
        L.sim_argmin.restype = C.c_int
        L.sim_best_reduce.argtypes = [P, P, I64, P, P]
        L.sim_best_reduce.restype = C.c_int
        L.sim_set_timing.argtypes = [P, C.c_int]
        L.sim_set_timing.restype = C.c_int
        L.sim_get_timing.argtypes = [P, C.c_int, C.POINTER(C.c_double), C.POINTER(I64)]
        L.sim_get_timing.restype = C.c_int
        L.sim_get_skipped_ops.argtypes = [P, C.POINTER(C.c_uint64)]
        L.sim_get_skipped_ops.restype = C.c_int
        L.sim_destroy.argtypes = [P]
        L.sim_destroy.restype = None
        L.sim_strerror.argtypes = [C.c_int]
        L.sim_strerror.restype = C.c_char_p
        _lib = L
    return _lib


class SimError(RuntimeError):
    def __init__(self, code, what):
        super().__init__("%s: %s (%d)" % (what, lib().sim_strerror(code).decode(), code))
        self.code = code


def _check(code, what):
    if code != SIM_OK:
        raise SimError(code, what)


def _u32(a):
    return np.ascontiguousarray(a, dtype=np.uint32)


def _u64(a):
    return np.ascontiguousarray(a, dtype=np.uint64)


def model_desc(m):
    """Pack a model dict into sim_model_desc; returns (desc, arrays kept alive)."""
    d = ModelDesc()
    d.n_layers, d.hidden, d.heads, d.kv_heads = m["L"], m["h"], m["heads"], m["kv_heads"]
    d.ffn, d.gated, d.vocab, d.learned_pos = m["ffn"], m["gated"], m["vocab"], m["learned_pos"]
    d.seq, d.dtype_bytes, d.global_batch = m["seq"], m["dtype_bytes"], m["global_batch"]
    d.n_mbs = len(m["mbs"])
    for i, v in enumerate(m["mbs"]):
        d.mbs[i] = v
    d.grad_bytes, d.param_bytes = m.get("grad_bytes", 4), m.get("param_bytes", 2)
    d.experts, d.topk, d.expert_ffn = m.get("experts", 0), m.get("topk", 0), m.get("expert_ffn", 0)
    d.opt_bytes = m.get("opt_bytes", 12)
    keep = []
    q = m.get("load_q16")
    if q is not None:
        qa = _u32(q)
        keep.append(qa)
        d.load_q16 = qa.ctypes.data
    return d, keep


def cluster_desc(c):
    d = ClusterDesc()
    d.n_types = len(c["types"])
    keep = []
    cols32 = ("n_nodes", "dev_per_node", "tflops", "hbm_GBps", "intra_MBps", "pcie_MBps", "nic_MBps")
    names32 = ("n_nodes", "dev_per_node", "tflops", "hbm_GBps", "intra_MBps", "pcie_MBps", "nic_MBps")
    for key, name in zip(cols32, names32):
        a = _u32([t[key] for t in c["types"]])
        keep.append(a)
        setattr(d, name, a.ctypes.data)
    for key in ("intra_alpha_ps", "pcie_alpha_ps", "nic_alpha_ps"):
        a = _u64([t[key] for t in c["types"]])
        keep.append(a)
        setattr(d, key, a.ctypes.data)
    for key in ("nic_MBps_dev", "intra_MBps_node"):
        if c.get(key) is not None:
            a = _u32(c[key])
            keep.append(a)
            setattr(d, key, a.ctypes.data)
    mem = [t.get("mem_bytes") for t in c["types"]]
    if any(v is not None for v in mem):
        a = _u64([v or 0 for v in mem])
        keep.append(a)
        d.mem_bytes = a.ctypes.data
    d.rail_only = 1 if c.get("rail_only") else 0
    d.ccl_tree = 1 if c.get("ccl_tree") else 0
    d.contention = 1 if c.get("contention") else 0
    d.ccl_hier = 1 if c.get("ccl_hier") else 0
    return d, keep


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def device_plans(p, device="cuda"):
    """Copy a host plan dict (numpy) to device tensors (bit-preserving int views).  A dict with
    chdr and ccut is a per-class-layout batch (its cut plane, if any, is not used)."""
    import torch
    d = dict(
        hdr=torch.from_numpy(np.ascontiguousarray(p["hdr"]).view(np.int32)).to(device),
        cls=torch.from_numpy(np.ascontiguousarray(p["cls"]).view(np.int32)).to(device),
        types=torch.from_numpy(np.ascontiguousarray(p["types"]).view(np.int64)).to(device),
    )
    if p.get("chdr") is not None:
        d["chdr"] = torch.from_numpy(np.ascontiguousarray(p["chdr"]).view(np.int32)).to(device)
        d["ccut"] = torch.from_numpy(np.ascontiguousarray(p["ccut"])).to(device)
    else:
        d["cut"] = torch.from_numpy(np.ascontiguousarray(p["cut"])).to(device)
    return d


def plans_struct(dp, offset=0):
    """sim_plans view of device plan tensors, starting at plan `offset`."""
    s = Plans()
    stride = dp["cls"].shape[1]
    s.hdr = dp["hdr"].data_ptr() + 4 * offset
    s.cls = dp["cls"].data_ptr() + 4 * offset
    s.types = dp["types"].data_ptr() + 8 * offset
    s.stride = stride
    if "chdr" in dp:
        assert dp["ccut"].shape == (64, stride)
        s.chdr = dp["chdr"].data_ptr() + 4 * offset
        s.ccut = dp["ccut"].data_ptr() + offset
    else:
        assert dp["cut"].shape == (16, stride)
        s.cut = dp["cut"].data_ptr() + offset
    return s


class Sim:
    """One evaluation context (model + cluster) on the current device."""

    def __init__(self, model, cluster):
        L = lib()
        md, k1 = model_desc(model)
        cd, k2 = cluster_desc(cluster)
        h = C.c_void_p()
        _check(L.sim_create(C.byref(md), C.byref(cd), C.byref(h)), "sim_create")
        self.h = h
        self._keep = (md, cd, k1, k2)

    def close(self):
        if getattr(self, "h", None):
            lib().sim_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def eval_plans(self, dp, n=None, out=None, offset=0, stream=None):
        """Iteration time (ps) of device plans [offset, offset+n) into an int64 tensor (uint64 bits)."""
        import torch
        if n is None:
            n = dp["hdr"].shape[0] - offset
        if out is None:
            out = torch.empty(n, dtype=torch.int64, device=dp["hdr"].device)
        ps = plans_struct(dp, offset)
        _check(lib().sim_eval_plans(self.h, C.byref(ps), n, out.data_ptr(), _stream(stream)), "sim_eval_plans")
        return out

    def eval_plans_noalloc(self, dp, n=None, out=None, offset=0, stream=None):
        """As eval_plans, through the allocation-free entry point (its workspace is the library's static
        device array; at most SIM_NOALLOC_MAX_PLANS plans per call).  `out` must be given: this call
        allocates nothing."""
        if n is None:
            n = dp["hdr"].shape[0] - offset
        assert out is not None, "eval_plans_noalloc writes into a caller-provided tensor"
        ps = plans_struct(dp, offset)
        _check(lib().sim_eval_plans_noalloc(self.h, C.byref(ps), n, out.data_ptr(), _stream(stream)),
               "sim_eval_plans_noalloc")
        return out

    def eval_stages(self, dp, n=None, stream=None):
        import torch
        if n is None:
            n = dp["hdr"].shape[0]
        st = torch.zeros((n, 4, 16, 4), dtype=torch.int64, device=dp["hdr"].device)
        cl = torch.zeros((n, 4), dtype=torch.int32, device=dp["hdr"].device)
        ps = plans_struct(dp)
        _check(lib().sim_eval_stages(self.h, C.byref(ps), n, st.data_ptr(), cl.data_ptr(), _stream(stream)),
               "sim_eval_stages")
        return st, cl

    def eval_memory(self, dp, n=None, stream=None):
        """Peak bytes per (class, stage) device: int64 tensor [n, 4, 16] (uint64 bits)."""
        import torch
        if n is None:
            n = dp["hdr"].shape[0]
        mem = torch.empty((n, 4, 16), dtype=torch.int64, device=dp["hdr"].device)
        ps = plans_struct(dp)
        _check(lib().sim_eval_memory(self.h, C.byref(ps), n, mem.data_ptr(), _stream(stream)), "sim_eval_memory")
        return mem

    def argmin(self, times, n=None, index_base=0, out=None, stream=None):
        """Lexicographic (time, index) minimum into a 2-word int64 tensor slot."""
        import torch
        if n is None:
            n = times.shape[0]
        if out is None:
            out = torch.empty(2, dtype=torch.int64, device=times.device)
        _check(lib().sim_argmin(self.h, times.data_ptr(), n, index_base, out.data_ptr(), _stream(stream)),
               "sim_argmin")
        return out

    def best_reduce(self, slots, out=None, stream=None):
        import torch
        if out is None:
            out = torch.empty(2, dtype=torch.int64, device=slots.device)
        n = slots.numel() // 2
        _check(lib().sim_best_reduce(self.h, slots.data_ptr(), n, out.data_ptr(), _stream(stream)),
               "sim_best_reduce")
        return out

    def set_timing(self, on):
        _check(lib().sim_set_timing(self.h, int(bool(on))), "sim_set_timing")

    def get_timing(self, kind):
        ms, cnt = C.c_double(), C.c_int64()
        _check(lib().sim_get_timing(self.h, kind, C.byref(ms), C.byref(cnt)), "sim_get_timing")
        return ms.value, cnt.value

    def get_skipped_ops(self):
        v = C.c_uint64()
        _check(lib().sim_get_skipped_ops(self.h, C.byref(v)), "sim_get_skipped_ops")
        return v.value


def measure_node_rate(stream=None):
    """Peak schedule-node rate of the current device (nodes/s; three fp64 VALU ops per node)."""
    v = C.c_double()
    _check(lib().sim_measure_node_rate(C.byref(v), _stream(stream)), "sim_measure_node_rate")
    return v.value


def best_tuple(slot_tensor):
    """(time_ps, index) of an argmin slot tensor."""
    a = slot_tensor.cpu().numpy()
    return int(a[0].view(np.uint64)), int(a[1])


def times_u64(t):
    return t.cpu().numpy().view(np.uint64)
