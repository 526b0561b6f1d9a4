"""Properties of the oracle's cluster options over seeded random configurations (the same
draws as the GPU parity cases), for every plan kind: no combination of options fails, none
changes which plans are valid, the tree and two-level all-reduces never make a plan slower
(each is taken only where faster), and rail-only forwarding and link contention never make a
plan faster (they only add hops or serialise link time)."""
import numpy as np
import pytest

from test_gpu_random_configs import OPTIONS, _config

MAXU = np.uint64(2**64 - 1)


def _kinds(workloads, m, c, s0, n):
    p = workloads.random_plans(m, c, s0, 0, n)
    kinds = {"plain": p}
    for kind, bit in (("overlap", 13), ("zero-bubble", 16)):
        q = {k: v.copy() for k, v in p.items()}
        q["hdr"] |= np.uint32(1 << bit)
        kinds[kind] = q
    kinds["interleaved"] = workloads.random_plans_il(m, c, s0 + 1, 0, n)
    kinds["per-class"] = workloads.random_plans_het(m, c, s0 + 2, 0, n)
    return kinds


@pytest.mark.parametrize("seed", range(16))
def test_option_monotonicity(oracle_mod, workloads, seed):
    _, m, c, s0 = _config(workloads, seed)
    base_c = dict(c, **{k: False for k in OPTIONS})
    base = oracle_mod.Oracle(m, base_c)
    for kind, q in _kinds(workloads, m, c, s0, 1200).items():
        t0 = base.eval(q)
        valid = t0 != MAXU
        for opt, faster in (("ccl_tree", True), ("ccl_hier", True), ("rail_only", False), ("contention", False)):
            t = oracle_mod.Oracle(m, dict(base_c, **{opt: True})).eval(q)
            assert np.array_equal(t != MAXU, valid), (seed, kind, opt)
            if faster:
                assert np.all(t[valid] <= t0[valid]), (seed, kind, opt)
            else:
                assert np.all(t[valid] >= t0[valid]), (seed, kind, opt)
        t = oracle_mod.Oracle(m, dict(base_c, **{k: True for k in OPTIONS})).eval(q)
        assert np.array_equal(t != MAXU, valid), (seed, kind, "all")
