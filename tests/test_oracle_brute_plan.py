"""Pin P8: the exhaustive 8-device workload evaluated by two independent evaluators.

oracle.c (max-plus recurrence, tabulated layer costs) and oracle/brute_plan.py (layer costs
rebuilt from the tensors each op moves, every pipeline replayed as a time-ordered event queue)
must give the same time for every one of the 29,470 plans, and so the same argmin.  A second
cluster splits each type's four devices over two nodes and adds a PCIe tier, so that hops and DP
rings take both the intra-node and the inter-node paths with PCIe latency on each end.
"""
import numpy as np
import pytest

from oracle import brute_plan


def _two_node_cluster(workloads):
    c = workloads.cluster_two_type_8()
    types = []
    for t, intra, pcie in zip(c["types"], (600_000, 200_000), (64_000, 32_000)):
        t = dict(t, n_nodes=2, dev_per_node=2, intra_MBps=intra, pcie_MBps=pcie, pcie_alpha_ps=143_750)
        types.append(t)
    return dict(c, types=types)


@pytest.mark.parametrize("cluster", ["one-node-per-type", "two-nodes-per-type-with-pcie"])
def test_exhaustive_workload_two_evaluators(oracle_mod, workloads, cluster):
    w = workloads.workload(1)
    c = w["cluster"] if cluster == "one-node-per-type" else _two_node_cluster(workloads)
    p = workloads.plans(w)
    want = oracle_mod.Oracle(w["model"], c).eval(p)
    ev = brute_plan.Plain(w["model"], c)
    got = np.array([ev.time(*brute_plan.plan_fields(p, i)) for i in range(p["hdr"].size)], dtype=np.uint64)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (cluster, bad[:5], got[bad[:5]], want[bad[:5]])
    assert int(np.argmin(got)) == int(np.argmin(want))
