"""Oracle of the front-end counts (TEST INFRASTRUCTURE ONLY: imported by the
test suite; the product package never imports it).

profiling_programs follows Sec. 4.3 (Eq. 2) by writing the programs out: one
program per strategy combination of the blocks of each distinct segment, and
one per strategy pair of every pair of blocks joined by a cross-segment
dependency.  Its length is the profiling-space size, counted by enumeration
rather than by the closed form.
"""
from __future__ import annotations

import itertools


def profiling_programs(strategies, deps=()):
    """Every program of the profiling space, as tuples:
    ("segment", i, (s_1, ..., s_K)) and ("reshard", entry, i, j, l, k, s_l, s_k)."""
    programs = []
    for i, seg in enumerate(strategies):
        for combo in itertools.product(*[range(s) for s in seg]):
            programs.append(("segment", i, combo))
    for entry, (i, j, l, k) in enumerate(deps):
        for s_l in range(strategies[i][l]):
            for s_k in range(strategies[j][k]):
                programs.append(("reshard", entry, i, j, l, k, s_l, s_k))
    return programs


def profiling_space_size(strategies, deps=()):
    return len(profiling_programs(strategies, list(deps)))
