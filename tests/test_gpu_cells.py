"""Per-layer costs measured from the kernels, and the cell split they give
(Sections 2.1-2.2), on the GPU.

The costs are measured step times, not values the oracle can compute
(parity unpinned); the checks are properties: every cost is positive, a
decoder layer (self-attention, cross-attention and feed-forward block) costs
more than an encoder layer of the same widths, and the least-variance split of
8 decoder layers and the 32000-way head into 3 cells leaves no cell further
from the mean cost than the largest single layer cost.
"""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu

pytest.importorskip("torch")


def test_measured_layer_costs_and_cells():
    from paper_1811_06965_amd import partitioner
    cfg = synth.CONFIGS["dec1024"]
    costs = partitioner.measure_layer_costs(cfg, steps=3, warmup=1)
    print("layer costs (ms per step):", costs)
    assert all(v > 0 for v in costs.values()), costs
    assert costs["decoder"] > costs["encoder"], costs
    kinds = ["decoder"] * 8 + ["head"]
    first, cell_costs, var = partitioner.plan(kinds, costs, 3)
    print("cells:", first, cell_costs, var)
    assert first[0] == 0 and sorted(first) == first and len(set(first)) == 3
    mean = sum(costs[k] for k in kinds) / 3
    assert max(abs(c - mean) for c in cell_costs) <= max(costs.values()), (cell_costs, mean)
    assert abs(np.var(cell_costs) - var) <= 1e-9 * max(1.0, var)
