"""Partitioning a sequence of layers into K cells, by exhaustive search.

TEST INFRASTRUCTURE ONLY (see the package docstring).

GPipe (Section 2.1) lets each layer i carry a cost estimate c_i; a cell p_k
of consecutive layers i..j costs C_k = sum_{l=i}^{j} c_l.  The partitioning
algorithm (Section 2.2) splits the L layers into K cells so that the variance
of the cell costs is minimal, which evens out the pipeline stages.

The variance is (1/K) sum_k (C_k - mean)^2 with mean = (sum_i c_i) / K fixed
by the costs, so this module enumerates every way of cutting the sequence
into K non-empty runs and keeps the one of least variance (ties: the
lexicographically smallest list of first layers).  Exponential in L: for
small cases only.
"""
from __future__ import annotations

import itertools
from typing import List, Sequence, Tuple


def cell_costs(costs: Sequence[float], first: Sequence[int]) -> List[float]:
    """C_k for cells starting at the layers in `first` (first[0] == 0)."""
    bounds = list(first) + [len(costs)]
    return [float(sum(costs[bounds[k]:bounds[k + 1]])) for k in range(len(first))]


def variance(costs: Sequence[float], first: Sequence[int]) -> float:
    C = cell_costs(costs, first)
    mean = sum(costs) / len(first)
    return sum((c - mean) ** 2 for c in C) / len(first)


def best_cells(costs: Sequence[float], K: int) -> Tuple[List[int], float]:
    """(first layer of every cell, variance) of the least-variance split of
    the layers into K non-empty cells of consecutive layers."""
    L = len(costs)
    if not 1 <= K <= L:
        raise ValueError("need 1 <= K <= number of layers")
    best, best_var = None, None
    for cuts in itertools.combinations(range(1, L), K - 1):
        first = [0, *cuts]
        v = variance(costs, first)
        if best_var is None or v < best_var:
            best, best_var = first, v
    return best, best_var
