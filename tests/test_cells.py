"""Partitioning a layer sequence into K cells of least cost variance
(Sections 2.1-2.2).

Pins of the exhaustive oracle (oracle/cells.py) against closed forms --
equal costs split into equal cells, one cell, one layer per cell, a cost
profile whose balanced split is known -- then the library's dynamic program
(gp_plan_cells, host code, no device) against the oracle on random costs,
and on the shapes of the paper's Transformer models (Table 1: up to 1663
layers, 128 cells), where the dynamic program must balance whole layers.
"""
import itertools
import os

import numpy as np
import pytest

from oracle import cells


def test_oracle_equal_costs_give_equal_cells():
    for L, K in ((12, 4), (12, 3), (8, 8), (9, 1)):
        first, var = cells.best_cells([2.5] * L, K)
        assert first == list(range(0, L, L // K)), (L, K, first)
        assert var == 0.0


def test_oracle_single_cell_and_one_layer_per_cell():
    c = [3.0, 1.0, 4.0, 1.0, 5.0]
    first, var = cells.best_cells(c, 1)
    assert first == [0]
    assert var == 0.0
    first, var = cells.best_cells(c, 5)
    assert first == [0, 1, 2, 3, 4]
    assert abs(var - np.var(c)) < 1e-14


def test_oracle_heavy_last_layer_gets_its_own_cell():
    """Decoder layers of cost 1 and a vocabulary head of cost 3 (about three
    layers): 9 layers + head into 4 cells -> three cells of three layers,
    the head alone, variance 0."""
    c = [1.0] * 9 + [3.0]
    first, var = cells.best_cells(c, 4)
    assert first == [0, 3, 6, 9]
    assert var == 0.0


def test_oracle_variance_definition():
    c = [1.0, 2.0, 3.0, 4.0]
    # cells [1,2] [3,4]: costs 3, 7, mean 5, variance 4
    assert cells.variance(c, [0, 2]) == 4.0
    assert cells.cell_costs(c, [0, 1, 3]) == [1.0, 5.0, 4.0]


@pytest.fixture(scope="module")
def gp():
    from paper_1811_06965_amd import build, gp as g
    if not os.path.exists(g.LIB_PATH):
        build.build()
    g.load()
    return g


def test_library_matches_exhaustive_search(gp):
    rng = np.random.default_rng(40)
    for trial in range(300):
        L = int(rng.integers(1, 11))
        K = int(rng.integers(1, L + 1))
        c = rng.uniform(0.1, 3.0, L)
        first, var = gp.gp_plan_cells(c, K)
        ref_first, ref_var = cells.best_cells(list(c), K)
        assert abs(var - ref_var) <= 1e-12 * max(1.0, ref_var), (L, K, var, ref_var)
        assert abs(cells.variance(list(c), first) - ref_var) <= 1e-12 * max(1.0, ref_var)
        # random real costs: the optimum is unique unless two splits tie to rounding
        if len({round(cells.variance(list(c), [0, *cuts]), 12)
                for cuts in itertools.combinations(range(1, L), K - 1)}) == \
                len(list(itertools.combinations(range(1, L), K - 1))):
            assert first == ref_first, (L, K, first, ref_first)


def test_library_balances_the_papers_largest_transformer(gp):
    """Transformer-1663 (Table 1's largest, 128 cells): equal layer costs
    split into cells of 12 or 13 layers; with a head of cost 2.6 layers the
    last cell takes fewer layers."""
    L, K = 1663, 128
    first, var = gp.gp_plan_cells(np.ones(L), K)
    sizes = np.diff(first + [L])
    assert set(sizes) == {12, 13} and sizes.sum() == L
    c = np.ones(L + 1)
    c[-1] = 2.6
    first, _ = gp.gp_plan_cells(c, K)
    assert np.diff(first + [L + 1])[-1] < 13


def test_library_rejects_bad_arguments(gp):
    with pytest.raises(gp.GpError) as e:
        gp.gp_plan_cells(np.ones(3), 4)
    assert e.value.status == gp.GP_ERR_INVALID_ARG
    with pytest.raises(gp.GpError):
        gp.gp_plan_cells(np.array([1.0, -1.0]), 1)
    with pytest.raises(gp.GpError):
        gp.gp_plan_cells(np.array([1.0, np.nan]), 2)
