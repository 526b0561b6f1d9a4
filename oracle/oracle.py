"""ctypes wrapper of the plain C oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: loaded by tests/, the smoke entry point and the CPU
baseline leg of the benchmark.  Takes plain dicts and numpy arrays so it shares
nothing with the HIP library's binding.
"""
import ctypes as C
import os

import numpy as np

from . import build as _build

_lib = None

OR_MAXG, OR_MAXS = 4, 16


class _Detail(C.Structure):
    _fields_ = [("valid", C.c_uint64), ("G", C.c_uint64),
                ("S", C.c_uint64 * OR_MAXG),
                ("M", C.c_uint64 * OR_MAXG),
                ("f", (C.c_uint64 * OR_MAXS) * OR_MAXG),
                ("b", (C.c_uint64 * OR_MAXS) * OR_MAXG),
                ("c", (C.c_uint64 * OR_MAXS) * OR_MAXG),
                ("w", (C.c_uint64 * OR_MAXS) * OR_MAXG),
                ("tdp", (C.c_uint64 * OR_MAXS) * OR_MAXG),
                ("end", (C.c_uint64 * OR_MAXS) * OR_MAXG),
                ("time", C.c_uint64)]


def lib():
    global _lib
    if _lib is None:
        # a mutated build of the same source may be named for tests that check the pins catch it
        path = os.environ.get("HETSIM_ORACLE_LIB") or _build.LIB
        if not os.path.exists(path):
            _build.build(force=False)
        L = C.CDLL(path)
        P = C.c_void_p
        u64 = C.c_uint64
        L.oracle_new.restype = P
        L.oracle_new.argtypes = [P, P, P, P, P]
        L.oracle_free.argtypes = [P]
        L.oracle_eval.argtypes = [P, P, P, P, P, P, P, C.c_int64, C.c_int64, P, C.c_int]
        L.oracle_detail.argtypes = [P, P, P, P, P, P, P, C.c_int64, C.c_int64, C.POINTER(_Detail)]
        L.oracle_detail.restype = C.c_int
        L.oracle_detail_size.restype = C.c_size_t
        L.oracle_pipeline.argtypes = [u64, u64, P, P, P, P]
        L.oracle_pipeline_interleaved.argtypes = [u64, u64, u64, P, P, P, u64, P]
        for name in ("oracle_alpha_ps", "oracle_beta_q"):
            getattr(L, name).argtypes = [u64]
            getattr(L, name).restype = u64
        L.oracle_link_time.argtypes = [u64, u64]
        L.oracle_link_time.restype = u64
        L.oracle_dp_sync.argtypes = [u64, u64, u64, u64, u64, u64]
        L.oracle_tree_allreduce.argtypes = [u64, u64, u64, u64]
        L.oracle_tree_allreduce.restype = u64
        L.oracle_hier_allreduce.argtypes = [u64] * 7
        L.oracle_hier_allreduce.restype = u64
        L.oracle_dp_sync.restype = u64
        L.oracle_layer_time.argtypes = [P, C.c_int, u64, u64, u64, u64, C.c_int]
        L.oracle_layer_time.restype = u64
        L.oracle_embed_time.argtypes = [P, C.c_int, u64, C.c_int]
        L.oracle_embed_time.restype = u64
        L.oracle_head_time.argtypes = [P, C.c_int, u64, u64, C.c_int]
        L.oracle_head_time.restype = u64
        L.oracle_param_count.argtypes = [P, C.c_int]
        L.oracle_param_count.restype = u64
        L.oracle_rank_params.argtypes = [P, u64, u64, u64]
        L.oracle_rank_params.restype = u64
        L.oracle_act_bytes.argtypes = [P, u64]
        L.oracle_act_bytes.restype = u64
        L.oracle_layer_act_bytes.argtypes = [P, u64, u64]
        L.oracle_layer_act_bytes.restype = u64
        L.oracle_in_flight.argtypes = [u64, u64, u64]
        L.oracle_in_flight.restype = u64
        L.oracle_in_flight_zb.argtypes = [u64, u64, u64]
        L.oracle_in_flight_zb.restype = u64
        L.oracle_pipeline_zb.argtypes = [u64, u64, P, P, P, P, P]
        L.oracle_stage_mem.argtypes = [P, P, P, P, P, P, P, C.c_int64, C.c_int64, P]
        L.oracle_stage_mem.restype = C.c_int
        assert L.oracle_detail_size() == C.sizeof(_Detail)
        _lib = L
    return _lib


def _ptr(a):
    return a.ctypes.data_as(C.c_void_p) if a is not None else None


MODEL_KEYS = ("L", "h", "heads", "kv_heads", "ffn", "gated", "vocab", "learned_pos", "seq",
              "dtype_bytes", "global_batch")


def _model_words(m):
    mbs = list(m["mbs"]) + [0] * (4 - len(m["mbs"]))
    w = [m[k] for k in MODEL_KEYS] + [len(m["mbs"])] + mbs + [
        m.get("grad_bytes", 4), m.get("param_bytes", 2), m.get("experts", 0), m.get("topk", 0),
        m.get("expert_ffn", 0), m.get("opt_bytes", 12)]
    return np.array(w, dtype=np.uint64)


TYPE_KEYS = ("n_nodes", "dev_per_node", "tflops", "hbm_GBps", "intra_MBps", "pcie_MBps", "nic_MBps",
             "intra_alpha_ps", "pcie_alpha_ps", "nic_alpha_ps")


def _cluster_words(c):
    w = [len(c["types"])]
    for t in c["types"]:
        w += [t[k] for k in TYPE_KEYS] + [t.get("mem_bytes") or 0]
    w.append(1 if c.get("rail_only") else 0)
    w.append(1 if c.get("ccl_tree") else 0)
    w.append(1 if c.get("contention") else 0)
    w.append(1 if c.get("ccl_hier") else 0)
    return np.array(w, dtype=np.uint64)


class Oracle:
    """CPU reference evaluator for one (model, cluster) pair."""

    def __init__(self, model, cluster):
        L = lib()
        self._mw = _model_words(model)
        self._cw = _cluster_words(cluster)
        q = model.get("load_q16")
        self._q = None if q is None else np.ascontiguousarray(q, dtype=np.uint32)
        nd = cluster.get("nic_MBps_dev")
        nn = cluster.get("intra_MBps_node")
        self._nd = None if nd is None else np.ascontiguousarray(nd, dtype=np.uint32)
        self._nn = None if nn is None else np.ascontiguousarray(nn, dtype=np.uint32)
        self.h = L.oracle_new(_ptr(self._mw), _ptr(self._q), _ptr(self._cw), _ptr(self._nd), _ptr(self._nn))

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.oracle_free(self.h)
            self.h = None

    @staticmethod
    def _planes(plans):
        """The plan planes as contiguous arrays; chdr/ccut only for the per-class layout."""
        hdr = np.ascontiguousarray(plans["hdr"], dtype=np.uint32)
        cls = np.ascontiguousarray(plans["cls"], dtype=np.uint32)
        typ = np.ascontiguousarray(plans["types"], dtype=np.uint64)
        stride = cls.shape[1]
        cut = plans.get("cut")
        cut = np.ascontiguousarray(cut, dtype=np.uint8) if cut is not None else None
        chdr = plans.get("chdr")
        ccut = plans.get("ccut")
        chdr = np.ascontiguousarray(chdr, dtype=np.uint32) if chdr is not None else None
        ccut = np.ascontiguousarray(ccut, dtype=np.uint8) if ccut is not None else None
        if cut is not None:
            assert cut.shape[1] == stride
        if ccut is not None:
            assert ccut.shape == (64, stride)
        return (hdr, cut, cls, typ, chdr, ccut), stride

    def eval(self, plans, nthreads=None, n=None):
        """plans: dict with hdr u32[n], cut u8[16, stride], cls u32[4, stride], types u64[4, stride], and for
        the per-class layout chdr u32[n] and ccut u8[64, stride] (cut may then be absent)."""
        arrs, stride = self._planes(plans)
        n = arrs[0].shape[0] if n is None else n
        out = np.empty(n, dtype=np.uint64)
        if nthreads is None:
            nthreads = os.cpu_count() or 1
        lib().oracle_eval(self.h, *[_ptr(a) for a in arrs], stride, n, _ptr(out), int(nthreads))
        return out

    def detail(self, plans, i):
        arrs, stride = self._planes(plans)
        d = _Detail()
        ok = lib().oracle_detail(self.h, *[_ptr(a) for a in arrs], stride, int(i), C.byref(d))
        if not ok:
            return None
        G = d.G
        S = [d.S[g] for g in range(G)]
        return {
            "S": S[0] if len(set(S)) == 1 else None, "S_class": S, "G": G, "M": [d.M[g] for g in range(G)],
            "f": [[d.f[g][s] for s in range(S[g])] for g in range(G)],
            "b": [[d.b[g][s] for s in range(S[g])] for g in range(G)],
            "c": [[d.c[g][s] for s in range(S[g])] for g in range(G)],
            "w": [[d.w[g][s] for s in range(S[g])] for g in range(G)],
            "tdp": [[d.tdp[g][s] for s in range(S[g])] for g in range(G)],
            "end": [[d.end[g][s] for s in range(S[g])] for g in range(G)],
            "time": d.time,
        }

    # pieces of the definition, exposed for pins
    def layer_time(self, k, t, b, ep, layer, bwd=False):
        return lib().oracle_layer_time(self.h, k, t, b, ep, layer, int(bwd))

    def embed_time(self, k, b, bwd=False):
        return lib().oracle_embed_time(self.h, k, b, int(bwd))

    def head_time(self, k, t, b, bwd=False):
        return lib().oracle_head_time(self.h, k, t, b, int(bwd))

    def param_count(self, with_head=True):
        return lib().oracle_param_count(self.h, int(with_head))

    def rank_params(self, t, ep, nlayers):
        return lib().oracle_rank_params(self.h, t, ep, nlayers)

    def act_bytes(self, b):
        return lib().oracle_act_bytes(self.h, b)

    def layer_act_bytes(self, t, b):
        return lib().oracle_layer_act_bytes(self.h, t, b)

    def stage_mem(self, plans, i):
        """[4][16] peak bytes per (class, stage) device of plan i, or None if a rule other than
        the memory check rejects the plan."""
        arrs, stride = self._planes(plans)
        mem = np.zeros((4, 16), dtype=np.uint64)
        ok = lib().oracle_stage_mem(self.h, *[_ptr(a) for a in arrs], stride, int(i), _ptr(mem))
        return mem if ok else None


def pipeline(S, M, f, b, c):
    """End time of each stage's last op for one 1F1B pipeline (c has S-1 hops)."""
    fa = np.array(f, dtype=np.uint64)
    ba = np.array(b, dtype=np.uint64)
    ca = np.array(list(c) + [0], dtype=np.uint64)
    end = np.zeros(S, dtype=np.uint64)
    lib().oracle_pipeline(S, M, _ptr(fa), _ptr(ba), _ptr(ca), _ptr(end))
    return [int(v) for v in end]


def pipeline_interleaved(S, v, M, f, b, c, cw):
    """End time of each device's last op for interleaved 1F1B: f, b per virtual stage (S*v), c the S-1
    hops between devices, cw the hop from the last device back to the first."""
    fa = np.array(f, dtype=np.uint64)
    ba = np.array(b, dtype=np.uint64)
    ca = np.array(list(c) + [0], dtype=np.uint64)
    end = np.zeros(S, dtype=np.uint64)
    lib().oracle_pipeline_interleaved(S, v, M, _ptr(fa), _ptr(ba), _ptr(ca), cw, _ptr(end))
    return [int(x) for x in end]


def in_flight(S, M, s):
    return lib().oracle_in_flight(S, M, s)


def in_flight_zb(S, M, s):
    return lib().oracle_in_flight_zb(S, M, s)


def pipeline_zb(S, M, f, bi, w, c):
    """End time of each stage's last op under the zero-bubble order: f, bi (input-gradient part
    of the backward) and w (weight-gradient part) per stage; c has S-1 hops."""
    arrs = [np.array(x, dtype=np.uint64) for x in (f, bi, w)]
    ca = np.array(list(c) + [0], dtype=np.uint64)
    end = np.zeros(S, dtype=np.uint64)
    lib().oracle_pipeline_zb(S, M, *[_ptr(a) for a in arrs], _ptr(ca), _ptr(end))
    return [int(x) for x in end]


def alpha_ps(gbps_unidir):
    return lib().oracle_alpha_ps(gbps_unidir)


def beta_q(MBps):
    return lib().oracle_beta_q(MBps)


def link_time(nbytes, bq):
    return lib().oracle_link_time(nbytes, bq)


def dp_sync(p, zero, grads, params, alpha, MBps):
    return lib().oracle_dp_sync(p, zero, grads, params, alpha, MBps)


def hier_allreduce(g, N, grads, a_in, MBps_in, alpha, MBps):
    return lib().oracle_hier_allreduce(g, N, grads, a_in, MBps_in, alpha, MBps)


def tree_allreduce(p, grads, alpha, MBps):
    return lib().oracle_tree_allreduce(p, grads, alpha, MBps)
