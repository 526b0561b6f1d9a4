"""Seeded synthetic workloads: model shapes, heterogeneous clusters and plans.

Input generation only (no time is computed here).  The five workloads mirror
the paper's setting: transformer models shaped like its Table 6 and the
public GPT-2/Llama/GPT-3 families, clusters of mixed device types with the
link tiers of its Table 5 (NVLink-class intra-node fabric, PCIe, RDMA NICs)
and interconnect delays from the jumbo-frame formula of Sec. 5.

Randomness is SplitMix64 used counter-based (see plangen.c); cluster seeds are
0xC1A50000 + config, plan seeds 0x91A70000 + config, expert-load seed
0xD1210004, device-memory seeds 0xC1A60000 + config.
"""
import ctypes as C
import itertools
import math
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(HERE, "plangen.c")
_LIB = os.path.join(HERE, "libplangen.so")
_lib = None

GOLDEN = 0x9E3779B97F4A7C15
M64 = (1 << 64) - 1


def build(force=True):
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-std=c11", "-Wall", "-fPIC", "-shared", "-pthread", _SRC, "-o", tmp],
                       check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Params(C.Structure):
    _fields_ = [("seed", C.c_uint64), ("L", C.c_uint32), ("K", C.c_uint32), ("cap", C.c_uint32 * 16),
                ("batches", C.c_uint32), ("experts", C.c_uint32)]


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = C.CDLL(_LIB)
        L.plangen_random.argtypes = [C.POINTER(_Params), C.c_uint64, C.c_int64, C.c_void_p, C.c_void_p,
                                     C.c_void_p, C.c_void_p, C.c_int64, C.c_int]
        L.plangen_random_het.argtypes = [C.POINTER(_Params), C.c_uint64, C.c_int64, C.c_void_p, C.c_void_p,
                                         C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_int]
        L.plangen_random_interleaved.argtypes = [C.POINTER(_Params), C.c_uint64, C.c_int64, C.c_void_p,
                                                 C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_int]
        L.plangen_draw.argtypes = [C.c_uint64, C.c_uint64]
        L.plangen_draw.restype = C.c_uint64
        _lib = L
    return _lib


def _mix(z):
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def draw(seed, counter):
    """SplitMix64 output number `counter` (0-based) of the stream starting at `seed`."""
    return _mix((seed + (counter + 1) * GOLDEN) & M64)


class Stream:
    def __init__(self, seed):
        self.seed, self.c = seed, 0

    def next(self):
        v = draw(self.seed, self.c)
        self.c += 1
        return v

    def uni(self, lo, hi):
        return lo + self.next() % (hi - lo + 1)

    def unit(self):
        """uniform double in (0, 1)"""
        return ((self.next() >> 11) + 0.5) / float(1 << 53)


# ---------------------------------------------------------------- links
def alpha_from_gbps(gbps_unidir):
    """Interconnect delay of one jumbo frame (9200 B) at a unidirectional rate, ps, rounded up."""
    return -(-9200 * 8 * 1000 // gbps_unidir)


def nic_MBps(gbps):
    return gbps * 125


# ---------------------------------------------------------------- models
MODELS = {
    "gpt2-small": dict(L=12, h=768, heads=12, kv_heads=12, ffn=3072, gated=0, vocab=50257, learned_pos=1024,
                       seq=1024, dtype_bytes=2, global_batch=8, mbs=[1]),
    "llama-7b": dict(L=32, h=4096, heads=32, kv_heads=32, ffn=11008, gated=1, vocab=32000, learned_pos=0,
                     seq=4096, dtype_bytes=2, global_batch=512, mbs=[1]),
    "llama-70b": dict(L=80, h=8192, heads=64, kv_heads=8, ffn=28672, gated=1, vocab=32000, learned_pos=0,
                      seq=4096, dtype_bytes=2, global_batch=1024, mbs=[1]),
    "mixtral-8x7b": dict(L=32, h=4096, heads=32, kv_heads=8, ffn=0, gated=1, vocab=32000, learned_pos=0,
                         seq=4096, dtype_bytes=2, global_batch=1152, mbs=[1], experts=8, topk=2,
                         expert_ffn=14336),
    "gpt3-175b": dict(L=96, h=12288, heads=96, kv_heads=96, ffn=49152, gated=0, vocab=50257, learned_pos=2048,
                      seq=2048, dtype_bytes=2, global_batch=1536, mbs=[1]),
}


def model(name, **over):
    m = dict(grad_bytes=4, param_bytes=2, opt_bytes=12, experts=0, topk=0, expert_ffn=0, load_q16=None)
    m.update(MODELS[name])
    m.update(over)
    return m


def dirichlet_q16(L, E, seed=0xD1210004):
    """Per-layer expert token shares ~ Dirichlet(1) (normalised -ln U), quantised to
    units of 2^-16 by largest remainder, ties to the lower expert."""
    st = Stream(seed)
    q = np.zeros((L, E), dtype=np.uint32)
    for l in range(L):
        g = [-math.log(st.unit()) for _ in range(E)]
        tot = sum(g)
        exact = [65536.0 * x / tot for x in g]
        base = [int(math.floor(x)) for x in exact]
        rem = 65536 - sum(base)
        order = sorted(range(E), key=lambda e: (-(exact[e] - base[e]), e))
        for e in order[:rem]:
            base[e] += 1
        q[l] = base
    return q


# ---------------------------------------------------------------- clusters
def _type(n_nodes, dpn, tflops, hbm, intra_MBps, pcie_MBps, nic, a_intra, a_pcie, a_nic):
    return dict(n_nodes=n_nodes, dev_per_node=dpn, tflops=tflops, hbm_GBps=hbm, intra_MBps=intra_MBps,
                pcie_MBps=pcie_MBps, nic_MBps=nic, intra_alpha_ps=a_intra, pcie_alpha_ps=a_pcie, nic_alpha_ps=a_nic)


def cluster_two_type_8():
    """8 devices: 4 of type A (312 TFLOPS, 2.0 TB/s) and 4 of type B (125 TFLOPS, 0.9 TB/s), one node each;
    300 GB/s intra-node, 25 GB/s inter-node, 2 us per hop (1 us per NIC side), no PCIe tier."""
    A = _type(1, 4, 312, 2000, 300_000, 0, 25_000, 2_000_000, 0, 1_000_000)
    B = _type(1, 4, 125, 900, 300_000, 0, 25_000, 2_000_000, 0, 1_000_000)
    return dict(types=[A, B], nic_MBps_dev=None, intra_MBps_node=None)


def cluster_fig3():
    """The two nodes of Sec. 3's worked example (Fig. 3): type 0 = node A, 4 x H100 80 GB; type 1 = node
    B, 4 x A100 40 GB.  Links and delays from Table 5 (its NVLink and PCIe rates are bidirectional
    totals, so half of each per direction; NIC 200 Gb/s with 368 ns processing; PCIe trips of 143.75
    and 287.5 ns).  The paper gives no device speeds: these are the public dense bf16 TFLOP/s and HBM
    GB/s of the two parts.  Memory capacities are not set (the example's Llama-2 70B does not fit
    four of these devices; give mem_bytes to check it)."""
    H100 = _type(1, 4, 989, 3350, 450_000, 64_000, nic_MBps(200), alpha_from_gbps(3600), 143_750, 368_000)
    A100 = _type(1, 4, 312, 1555, 300_000, 32_000, nic_MBps(200), alpha_from_gbps(2400), 287_500, 368_000)
    return dict(types=[H100, A100], nic_MBps_dev=None, intra_MBps_node=None)


def cluster_random(cfg, nodes, dpn=8, nic_choices=(100, 200, 400), pcie=True, jitter=False, pcie_only_types=(),
                   alpha_mult=False):
    st = Stream(0xC1A50000 + cfg)
    types = []
    for k, n in enumerate(nodes):
        tflops = st.uni(100, 1000)
        hbm = st.uni(900, 8000)
        intra_GBps = st.uni(300, 900)
        gbps = nic_choices[st.uni(0, len(nic_choices) - 1)]
        if k in pcie_only_types:
            intra, a_intra = 64_000, 2 * 143_750
        else:
            intra, a_intra = intra_GBps * 1000, alpha_from_gbps(intra_GBps * 8)
        if alpha_mult:
            a_intra *= st.uni(1, 4)
        types.append(_type(n, dpn, tflops, hbm, intra, 64_000 if pcie else 0, nic_MBps(gbps), a_intra,
                           143_750 if pcie else 0, alpha_from_gbps(gbps)))
    c = dict(types=types, nic_MBps_dev=None, intra_MBps_node=None)
    if jitter:
        dev, node = [], []
        for t in types:
            for _ in range(t["n_nodes"] * t["dev_per_node"]):
                dev.append(t["nic_MBps"] * st.uni(800, 1200) // 1000)
            for _ in range(t["n_nodes"]):
                node.append(t["intra_MBps"] * st.uni(800, 1200) // 1000)
        c["nic_MBps_dev"] = np.array(dev, dtype=np.uint32)
        c["intra_MBps_node"] = np.array(node, dtype=np.uint32)
    return c


# device memory sizes of accelerators of the last generations, GiB (Table 5's
# A100 40 GB and H100 80 GB among them)
MEM_GIB = (16, 24, 32, 40, 48, 64, 80, 96, 128, 141, 192, 288)


def with_memory(w, gib=None):
    """Copy of workload w whose device types have a memory capacity: `gib` per type, or drawn per type
    from MEM_GIB with the seed 0xC1A60000 + the workload's index."""
    types = [dict(t) for t in w["cluster"]["types"]]
    if gib is None:
        st = Stream(0xC1A60000 + w["index"])
        gib = [MEM_GIB[st.uni(0, len(MEM_GIB) - 1)] for _ in types]
    for t, g in zip(types, gib):
        t["mem_bytes"] = int(g) << 30
    return dict(w, name=w["name"] + "/mem", cluster=dict(w["cluster"], types=types))


# ---------------------------------------------------------------- plans
def empty_plans(n):
    return dict(hdr=np.zeros(n, np.uint32), cut=np.zeros((16, n), np.uint8), cls=np.zeros((4, n), np.uint32),
                types=np.zeros((4, n), np.uint64))


def random_plans(m, c, seed, first, n, nthreads=None, out=None):
    """Plans first..first+n-1 of the seeded random generator (see plangen.c)."""
    L = _load()
    P = _Params()
    P.seed = seed
    P.L = m["L"]
    P.K = len(c["types"])
    for k, t in enumerate(c["types"]):
        P.cap[k] = t["n_nodes"] * t["dev_per_node"]
    P.batches = m["global_batch"] // m["mbs"][0]
    P.experts = m.get("experts", 0)
    p = empty_plans(n) if out is None else out
    stride = p["cut"].shape[1]
    if nthreads is None:
        nthreads = min(16, os.cpu_count() or 1)
    L.plangen_random(C.byref(P), first, n, p["hdr"].ctypes.data, p["cut"].ctypes.data, p["cls"].ctypes.data,
                     p["types"].ctypes.data, stride, nthreads)
    return p


def random_plans_het(m, c, seed, first, n, nthreads=None):
    """Per-class-layout plans first..first+n-1 (every class its own TP degree, pipeline depth and layer
    split; see plangen.c): dict with hdr, cls, types, chdr (u32 [n]) and ccut (u8 [64, n])."""
    L = _load()
    P = _Params()
    P.seed = seed
    P.L = m["L"]
    P.K = len(c["types"])
    for k, t in enumerate(c["types"]):
        P.cap[k] = t["n_nodes"] * t["dev_per_node"]
    P.batches = m["global_batch"] // m["mbs"][0]
    P.experts = m.get("experts", 0)
    p = dict(hdr=np.zeros(n, np.uint32), cls=np.zeros((4, n), np.uint32), types=np.zeros((4, n), np.uint64),
             chdr=np.zeros(n, np.uint32), ccut=np.zeros((64, n), np.uint8))
    if nthreads is None:
        nthreads = min(16, os.cpu_count() or 1)
    L.plangen_random_het(C.byref(P), first, n, p["hdr"].ctypes.data, p["ccut"].ctypes.data, p["cls"].ctypes.data,
                         p["types"].ctypes.data, p["chdr"].ctypes.data, n, nthreads)
    return p


def random_plans_il(m, c, seed, first, n, nthreads=None):
    """Interleaved-1F1B plans (see plangen.c): v = 2..4 model chunks per device, S devices with
    S*v <= 16, every class's micro-batches per replica a multiple of S and at least 2S."""
    L = _load()
    P = _Params()
    P.seed = seed
    P.L = m["L"]
    P.K = len(c["types"])
    for k, t in enumerate(c["types"]):
        P.cap[k] = t["n_nodes"] * t["dev_per_node"]
    P.batches = m["global_batch"] // m["mbs"][0]
    P.experts = m.get("experts", 0)
    p = empty_plans(n)
    if nthreads is None:
        nthreads = min(16, os.cpu_count() or 1)
    L.plangen_random_interleaved(C.byref(P), first, n, p["hdr"].ctypes.data, p["cut"].ctypes.data,
                                 p["cls"].ctypes.data, p["types"].ctypes.data, n, nthreads)
    return p


def interleaved_plans(w, first=0, n=None, nthreads=None):
    """Interleaved plans of workload w (its own seed + 0x200)."""
    if n is None:
        n = w["n_plans"] - first
    seed = (w["seed"] if w["seed"] is not None else 0x91A70001) + 0x200
    return random_plans_il(w["model"], w["cluster"], seed, first, n, nthreads)


def as_per_class(p):
    """The per-class-layout encoding of shared-layout plans: every class gets the plan's TP degree, depth,
    micro-batch size and cuts (header TP, PP and micro-batch size fields cleared)."""
    n = p["hdr"].shape[0]
    hdr = p["hdr"].astype(np.uint32)
    tpl = hdr & 3
    pp1 = (hdr >> 4) & 15
    G = ((hdr >> 8) & 3) + 1
    mi = (hdr >> 11) & 3
    chdr = np.zeros(n, np.uint32)
    ccut = np.zeros((64, n), np.uint8)
    for c in range(4):
        has = G > c
        chdr |= np.where(has, (tpl | (pp1 << 2) | (mi << 6)) << (8 * c), 0).astype(np.uint32)
        ccut[c * 16:(c + 1) * 16] = np.where(has[None, :], p["cut"][:, :n], 0)
    return dict(hdr=hdr & ~np.uint32(0x18F3), cls=np.ascontiguousarray(p["cls"][:, :n]),
                types=np.ascontiguousarray(p["types"][:, :n]), chdr=chdr, ccut=ccut)


def het_plans(w, first=0, n=None, nthreads=None):
    """Per-class-layout plans of workload w (its own seed + 0x100)."""
    if n is None:
        n = w["n_plans"] - first
    seed = (w["seed"] if w["seed"] is not None else 0x91A70001) + 0x100
    return random_plans_het(w["model"], w["cluster"], seed, first, n, nthreads)


def enumerate_two_type_8(L=12, n_dev=8, per_type=4, batches=8):
    """Every plan of the 8-device two-type cluster with TP 1: PP in {1,2,4,8}, DP = 8/PP,
    every contiguous split of the L layers, every assignment of device types to the
    DP x PP (replica, stage) slots using 4 of each type, up to permuting replicas.
    Replicas with the same type vector form one class; each replica runs
    batches/DP micro-batches.  Order: PP, then cut points (lexicographic), then the
    sorted tuple of replica type vectors (lexicographic; bit s set = type B)."""
    rows = []
    for pp in (1, 2, 4, 8):
        dp = n_dev // pp
        splits = list(itertools.combinations(range(1, L), pp - 1))
        assigns = []
        for combo in itertools.combinations_with_replacement(range(1 << pp), dp):
            n_b = sum(bin(v).count("1") for v in combo)
            if n_b != per_type:
                continue
            assigns.append(combo)
        for sp in splits:
            cuts = list(sp) + [L]
            for combo in assigns:
                classes = []
                for v in combo:
                    if classes and classes[-1][0] == v:
                        classes[-1][1] += 1
                    else:
                        classes.append([v, 1])
                rows.append((pp, cuts, classes, batches // dp))
    n = len(rows)
    p = empty_plans(n)
    for i, (pp, cuts, classes, per_rep) in enumerate(rows):
        G = len(classes)
        p["hdr"][i] = ((pp - 1) << 4) | ((G - 1) << 8)
        for s, v in enumerate(cuts):
            p["cut"][s, i] = v
        for g, (v, reps) in enumerate(classes):
            p["cls"][g, i] = reps | ((reps * per_rep) << 16)
            t = 0
            for s in range(pp):
                t |= ((v >> s) & 1) << (4 * s)
            p["types"][g, i] = t
    return p


# ---------------------------------------------------------------- the five workloads
def workload(idx):
    """Workload idx in 1..5: dict(name, model, cluster, n_plans, seed)."""
    if idx == 1:
        return dict(index=1, name="gpt2-small/8dev-2type/exhaustive", model=model("gpt2-small"),
                    cluster=cluster_two_type_8(), n_plans=29470, seed=None)
    if idx == 2:
        return dict(index=2, name="llama-7b/64dev-3type/1M", model=model("llama-7b"),
                    cluster=cluster_random(2, [3, 3, 2]), n_plans=1 << 20, seed=0x91A70002)
    if idx == 3:
        return dict(index=3, name="llama-70b/512dev-4type-jitter/16M", model=model("llama-70b"),
                    cluster=cluster_random(3, [16, 16, 16, 16], nic_choices=(200, 400), pcie=False, jitter=True),
                    n_plans=1 << 24, seed=0x91A70003)
    if idx == 4:
        m = model("mixtral-8x7b")
        m["load_q16"] = dirichlet_q16(m["L"], m["experts"])
        return dict(index=4, name="mixtral-8x7b/256dev-3type/4M", model=m, cluster=cluster_random(4, [11, 11, 10]),
                    n_plans=1 << 22, seed=0x91A70004)
    if idx == 5:
        return dict(index=5, name="gpt3-175b/4096dev-6type-3tier/64M", model=model("gpt3-175b"),
                    cluster=cluster_random(5, [86, 86, 85, 85, 85, 85], pcie_only_types=(4, 5), alpha_mult=True),
                    n_plans=1 << 26, seed=0x91A70005)
    raise ValueError(idx)


def plans(w, first=0, n=None, nthreads=None):
    """Plans [first, first+n) of workload dict w."""
    if n is None:
        n = w["n_plans"] - first
    if w["seed"] is None:
        p = enumerate_two_type_8()
        return {k: (v[first:first + n] if k == "hdr" else np.ascontiguousarray(v[:, first:first + n]))
                for k, v in p.items()}
    return random_plans(w["model"], w["cluster"], w["seed"], first, n, nthreads)
