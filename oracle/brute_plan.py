"""A second, independent whole-plan evaluator, for the plain 1F1B plans of dense models at TP 1.

TEST INFRASTRUCTURE ONLY (tests/ import it; nothing in the product does).  Written from the
readings of the paper that the oracle also follows, but sharing no code with oracle.c: it
rebuilds each layer's cost from the tensors its ops read and write, places the devices, prices
the hops and the DP ring, and replays every pipeline with the time-ordered event simulator of
brute_sim.py instead of the max-plus recurrence.  Slow; meant for the 8-device exhaustive
workload (29,470 plans), where it checks every time and the argmin against the oracle.

Scope (anything else raises): shared layout, TP 1, EP 1, no ZeRO, no overlap, no interleaving,
no zero-bubble order, no cluster options, no device-memory check, no per-device or per-node
rates.

Readings used (both evaluators implement them):
  time is integer ps and every division rounds up; an op takes the longer of its FLOPs at the
  device's TFLOP/s and its bytes at its HBM GB/s; a backward op costs twice its forward FLOPs and
  bytes; a GEMM [m x k][k x n] does 2mkn FLOPs and moves its three matrices; attention counts
  4 b s^2 h FLOPs (non-causal) and moves Q, K, V and O; the vocabulary is padded to a multiple of
  128; a link moves a byte in ceil(2^16 * 10^6 / MB/s) / 2^16 ps; an inter-node endpoint costs two
  PCIe trips plus the NIC; PP messages carry one micro-batch's activation; gradients are fp32 and
  sync in a ring over every replica after the last backward pass.
"""
from . import brute_sim

Q = 1 << 16


def cdiv(a, b):
    return -(-a // b)


def beta(MBps):
    """Link time per byte in units of 2^-16 ps; 0 = no such link."""
    return cdiv(Q * 10**6, MBps) if MBps else 0


def move(nbytes, bq):
    return cdiv(nbytes * bq, Q)


class Device:
    """One device type's speed."""

    def __init__(self, t):
        self.tflops, self.hbm = t["tflops"], t["hbm_GBps"]

    def op(self, flops, nbytes):
        return max(cdiv(flops, self.tflops), cdiv(1000 * nbytes, self.hbm))


def _gemm(m, k, n, e):
    """(FLOPs, bytes) of [m x k] @ [k x n] -> [m x n]."""
    return 2 * m * k * n, e * (m * k + k * n + m * n)


class Plain:
    def __init__(self, model, cluster):
        m = self.m = model
        if m.get("experts") or m.get("gated"):
            raise ValueError("dense, non-gated models only")
        self.types = cluster["types"]
        if cluster.get("nic_MBps_dev") is not None or cluster.get("intra_MBps_node") is not None:
            raise ValueError("no per-device or per-node rates")
        for opt in ("rail_only", "ccl_tree", "contention", "ccl_hier"):
            if cluster.get(opt):
                raise ValueError("no cluster options")
        if any(t.get("mem_bytes") for t in self.types):
            raise ValueError("no memory check")
        self.dev = [Device(t) for t in self.types]
        self.Vp = cdiv(m["vocab"], 128) * 128
        self._cost = {}

    # ---- compute
    def _layer_ops(self, b):
        """(FLOPs, bytes) of each op of one transformer layer for b sequences, TP 1."""
        m = self.m
        e, h, s, f = m["dtype_bytes"], m["h"], m["seq"], m["ffn"]
        T = b * s
        kvw = m["kv_heads"] * (h // m["heads"])     # width of K and of V
        act = T * h * e                             # one [T x h] tensor
        return [
            (0, 2 * act),                           # norm: read x, write y
            _gemm(T, h, h + 2 * kvw, e),            # Q, K, V projection
            (4 * b * s * s * h, e * T * (h + 2 * kvw) + e * T * h),   # attention: read Q, K, V; write O
            _gemm(T, h, h, e),                      # output projection
            (0, 3 * act),                           # residual: read two, write one
            (0, 2 * act),                           # norm
            _gemm(T, h, f, e),                      # MLP up
            (0, 2 * T * f * e),                     # activation: read, write
            _gemm(T, f, h, e),                      # MLP down
            (0, 3 * act),                           # residual
        ]

    def _embed_ops(self, b):
        m = self.m
        T = b * m["seq"]
        per_token = 2 + (2 if m["learned_pos"] else 0)    # read the row and write it; positions: read, add
        return [(0, m["dtype_bytes"] * T * m["h"] * per_token)]

    def _head_ops(self, b):
        m = self.m
        e, h, T = m["dtype_bytes"], m["h"], b * m["seq"]
        return [(0, 2 * T * h * e), _gemm(T, h, self.Vp, e), (0, 2 * T * self.Vp * e)]

    def _time(self, k, ops, bwd):
        d = self.dev[k]
        return sum(d.op(2 * F if bwd else F, 2 * B if bwd else B) for F, B in ops)

    def stage_time(self, k, lo, hi, first, last, b):
        """(forward, backward) of one micro-batch over layers [lo, hi) on type k."""
        key = (k, lo, hi, first, last, b)
        if key not in self._cost:
            ops = self._layer_ops(b) * (hi - lo)
            if first:
                ops = ops + self._embed_ops(b)
            if last:
                ops = ops + self._head_ops(b)
            self._cost[key] = (self._time(k, ops, False), self._time(k, ops, True))
        return self._cost[key]

    # ---- links
    def _side(self, k):
        t = self.types[k]
        return 2 * t["pcie_alpha_ps"] + t["nic_alpha_ps"]

    def _node(self, k, d):
        return d // self.types[k]["dev_per_node"]

    def hop(self, k1, b1, k2, b2, reps, act):
        """Pipeline hop between the stage on devices [b1, b1+reps) of pool k1 and [b2, ...) of k2."""
        same_node = k1 == k2 and all(self._node(k1, b1 + r) == self._node(k2, b2 + r) for r in range(reps))
        if same_node:
            return self.types[k1]["intra_alpha_ps"] + move(act, beta(self.types[k1]["intra_MBps"]))
        bq = max(beta(self.types[k]["nic_MBps"]) for k in (k1, k2))
        bq = max(bq, max(beta(self.types[k]["pcie_MBps"]) for k in (k1, k2)))
        return self._side(k1) + self._side(k2) + move(act, bq)

    def dp(self, members, nbytes):
        """Ring all-reduce of nbytes per member over the devices `members` [(type, device)]."""
        p = len(members)
        if p <= 1:
            return 0
        nodes = {(k, self._node(k, d)) for k, d in members}
        if len(nodes) == 1:
            k = members[0][0]
            alpha, bq = self.types[k]["intra_alpha_ps"], beta(self.types[k]["intra_MBps"])
        else:
            ks = {k for k, _ in members}
            alpha = max(2 * self._side(k) for k in ks)
            bq = max(max(beta(self.types[k]["nic_MBps"]), beta(self.types[k]["pcie_MBps"])) for k in ks)
        steps = 2 * (p - 1)
        return steps * alpha + move(steps * cdiv(nbytes, p), bq)

    def params(self, lo, hi, first, last):
        m = self.m
        h, f = m["h"], m["ffn"]
        kvw = m["kv_heads"] * (h // m["heads"])
        layer = h * (h + 2 * kvw) + h * h + 2 * h + 2 * h * f
        n = (hi - lo) * layer
        if first:
            n += self.Vp * h + m["learned_pos"] * h
        if last:
            n += self.Vp * h + h
        return n

    # ---- one plan
    def time(self, hdr, cuts, classes):
        """hdr: the plan's header word; cuts: cumulative stage ends; classes: [(reps, nmb, [type per
        stage])].  Returns the iteration time in ps."""
        m = self.m
        if hdr & ~((15 << 4) | (3 << 8) | (3 << 11)):
            raise ValueError("plain plans at TP 1 without ZeRO only")
        S = len(cuts)
        b = m["mbs"][(hdr >> 11) & 3]
        act = b * m["seq"] * m["h"] * m["dtype_bytes"]
        # placement: each pool is filled in (class, stage) order, reps devices per stage
        nxt = [0] * len(self.types)
        base = []
        for reps, _, ty in classes:
            row = []
            for s in range(S):
                row.append(nxt[ty[s]])
                nxt[ty[s]] += reps
            base.append(row)
        for k, t in enumerate(self.types):
            if nxt[k] > t["n_nodes"] * t["dev_per_node"]:
                raise ValueError("does not fit")
        ends = []
        for g, (reps, nmb, ty) in enumerate(classes):
            f, bw, c = [], [], []
            lo = 0
            for s in range(S):
                ff, bb = self.stage_time(ty[s], lo, cuts[s], s == 0, s == S - 1, b)
                f.append(ff)
                bw.append(bb)
                if s > 0:
                    c.append(self.hop(ty[s - 1], base[g][s - 1], ty[s], base[g][s], reps, act))
                lo = cuts[s]
            c.append(0)
            M = cdiv(nmb, reps)
            end, _ = brute_sim.simulate(S, M, f, bw, c)
            ends.append(end)
        T = 0
        lo = 0
        for s in range(S):
            members = [(ty[s], base[g][s] + r) for g, (reps, _, ty) in enumerate(classes) for r in range(reps)]
            sync = self.dp(members, m["grad_bytes"] * self.params(lo, cuts[s], s == 0, s == S - 1))
            T = max(T, max(e[s] for e in ends) + sync)
            lo = cuts[s]
        return T


def plan_fields(p, i):
    """(hdr, cuts, classes) of plan i of the shared-layout planes p."""
    hdr = int(p["hdr"][i])
    S = ((hdr >> 4) & 15) + 1
    G = ((hdr >> 8) & 3) + 1
    cuts = [int(p["cut"][s, i]) for s in range(S)]
    classes = []
    for g in range(G):
        w = int(p["cls"][g, i])
        tv = int(p["types"][g, i])
        classes.append((w & 0xFFFF, w >> 16, [(tv >> (4 * s)) & 15 for s in range(S)]))
    return hdr, cuts, classes
