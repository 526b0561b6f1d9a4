"""The seeded input generators shared by the HIP path and the oracle."""
import hashlib

import numpy as np


def test_splitmix64_known_answers(workloads):
    # SplitMix64 from state 0 (Steele, Lea, Flood 2014): first three outputs
    assert workloads.draw(0, 0) == 0xE220A8397B1DCDAF
    assert workloads.draw(0, 1) == 0x6E789E6AA1B965F4
    assert workloads.draw(0, 2) == 0x06C45D188009454F
    # the C generator uses the same stream
    L = workloads._load()
    for s, c in ((0, 0), (12345, 99), (0x91A70003, 4096 * 7 + 5)):
        assert L.plangen_draw(s, c) == workloads.draw(s, c)


def test_exhaustive_two_type_count(workloads):
    p = workloads.enumerate_two_type_8()
    hdr = p["hdr"]
    pp = ((hdr >> 4) & 15) + 1
    # splits C(11, pp-1) times type multisets with four devices of each type
    assert len(hdr) == 29470
    assert [(pp == k).sum() for k in (1, 2, 4, 8)] == [1, 99, 6270, 23100]
    G = ((hdr >> 8) & 3) + 1
    reps = p["cls"] & 0xFFFF
    nmb = p["cls"] >> 16
    for i in range(0, len(hdr), 997):
        g = G[i]
        assert reps[:g, i].sum() * pp[i] == 8
        assert nmb[:g, i].sum() == 8
        # four devices of each type
        nb = 0
        for c in range(g):
            tv = int(p["types"][c, i])
            nb += reps[c, i] * sum((tv >> (4 * s)) & 1 for s in range(pp[i]))
        assert nb == 4


def _digest(p):
    h = hashlib.sha256()
    for k in ("hdr", "cut", "cls", "types"):
        h.update(np.ascontiguousarray(p[k]).tobytes())
    return h.hexdigest()


def test_random_plans_deterministic_and_chunkable(workloads):
    w = workloads.workload(3)
    a = workloads.plans(w, 0, 5000, nthreads=1)
    b = workloads.plans(w, 0, 5000, nthreads=7)
    assert _digest(a) == _digest(b)
    c = workloads.plans(w, 2000, 1000)
    assert np.array_equal(c["hdr"], a["hdr"][2000:3000])
    assert np.array_equal(c["cut"], a["cut"][:, 2000:3000])


def test_random_plans_structure(workloads):
    for idx in (2, 3, 4, 5):
        w = workloads.workload(idx)
        p = workloads.plans(w, 0, 4000)
        hdr = p["hdr"]
        assert np.all(hdr >> 13 == 0)
        S = ((hdr >> 4) & 15) + 1
        G = ((hdr >> 8) & 3) + 1
        L = w["model"]["L"]
        for i in range(0, 4000, 37):
            cuts = p["cut"][: S[i], i].astype(int)
            assert cuts[-1] == L and np.all(np.diff(cuts) > 0) and cuts[0] >= 1
            nmb = (p["cls"][: G[i], i] >> 16).sum()
            assert nmb == w["model"]["global_batch"]


def test_dirichlet_loads(workloads):
    q = workloads.dirichlet_q16(32, 8)
    assert q.shape == (32, 8) and np.all(q.sum(1) == 65536)
    assert len({tuple(r) for r in q}) == 32            # layers differ
    assert q.min() < 65536 // 8 < q.max()               # imbalanced


def test_cluster_shapes(workloads):
    for idx, ndev in ((1, 8), (2, 64), (3, 512), (4, 256), (5, 4096)):
        c = workloads.workload(idx)["cluster"]
        assert sum(t["n_nodes"] * t["dev_per_node"] for t in c["types"]) == ndev
    c = workloads.workload(3)["cluster"]
    assert len(c["nic_MBps_dev"]) == 512 and len(c["intra_MBps_node"]) == 64
    assert all(t["pcie_MBps"] == 0 for t in c["types"])
