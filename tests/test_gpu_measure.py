"""The node-rate probe that bench.py uses for its roofline peak."""
import pytest

pytestmark = pytest.mark.gpu


def test_node_rate_probe_is_below_issue_rate():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_05370_amd import binding as B
    rate = B.measure_node_rate()
    spec = 256 * 64 * 2.4e9                  # VALU lane-ops per second, one instruction per lane per clock
    # a node is three fp64 VALU instructions; the probe cannot issue faster than the chip
    assert 0.2 * spec / 3 < rate <= 1.05 * spec / 3, rate
