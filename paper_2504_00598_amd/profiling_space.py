"""Size of the profiling space (Sec. 4.3, Eq. 2): how many parallel programs
must be compiled and profiled before the plan search can run.

A model has N distinct segments; segment i holds K_i ParallelBlocks and block
j of segment i has S_{i,j} parallel strategies.  Every strategy combination of
the blocks of a segment is one program (the product over j of S_{i,j}), and
every pair of blocks (l of segment i, k of segment j) joined by a
cross-segment tensor dependency needs one resharding program per pair of their
strategies (S_{i,l} * S_{j,k}).  The count is the sum of both parts over all
segments and all dependent pairs (the pair list of segments i and j is D_{i,j}).

This is host-side bookkeeping: no part of it runs on the GPU.
"""
from __future__ import annotations

from typing import Iterable, Sequence, Tuple

Dependency = Tuple[int, int, int, int]  # (i, j, l, k): block l of segment i and block k of segment j


def _check(strategies: Sequence[Sequence[int]], deps: Sequence[Dependency]) -> None:
    if not strategies:
        raise ValueError("at least one segment")
    for i, seg in enumerate(strategies):
        if not seg:
            raise ValueError(f"segment {i} has no ParallelBlock")
        for s in seg:
            if int(s) != s or s < 1:
                raise ValueError(f"segment {i}: strategy counts are positive integers, got {s!r}")
    for dep in deps:
        if len(dep) != 4:
            raise ValueError(f"a dependency is (i, j, l, k), got {dep!r}")
        i, j, l, k = dep
        if not (0 <= i < len(strategies) and 0 <= j < len(strategies)):
            raise ValueError(f"dependency {dep!r}: no such segment")
        if not (0 <= l < len(strategies[i]) and 0 <= k < len(strategies[j])):
            raise ValueError(f"dependency {dep!r}: no such ParallelBlock")


def segment_plans(strategies_of_segment: Sequence[int]) -> int:
    """Programs of one segment: the product of its blocks' strategy counts."""
    n = 1
    for s in strategies_of_segment:
        n *= int(s)
    return n


def profiling_space_size(strategies: Sequence[Sequence[int]], deps: Iterable[Dependency] = ()) -> int:
    """Eq. 2: sum over segments of the segment's plan count, plus
    S_{i,l} * S_{j,k} for every listed dependency (i, j, l, k), 0-based.  A
    dependency listed twice is counted twice, as a list entry of D_{i,j}."""
    deps = list(deps)
    _check(strategies, deps)
    total = sum(segment_plans(seg) for seg in strategies)
    total += sum(int(strategies[i][l]) * int(strategies[j][k]) for i, j, l, k in deps)
    return total
