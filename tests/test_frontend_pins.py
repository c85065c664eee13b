"""The profiling-space count (Sec. 4.3, Eq. 2) against the oracle's
enumeration of every program, pinned by the paper's printed example (Sec. 5.5:
180 programs for GPT-like models) and by the worst and best cases Sec. 4.3
states in closed form."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

from oracle import frontend as OF
from paper_2504_00598_amd.profiling_space import profiling_space_size, segment_plans

HERE = os.path.dirname(os.path.abspath(__file__))


def test_printed_example_180():
    with open(os.path.join(HERE, "golden", "profiling_space_gpt.json")) as f:
        g = json.load(f)
    deps = [tuple(d) for d in g["deps"]]
    assert OF.profiling_space_size(g["strategies"], deps) == g["total"] == 180
    assert profiling_space_size(g["strategies"], deps) == 180


def test_worst_case_single_segment():
    """The whole model as one distinct segment of M blocks: the product of the
    strategy counts, as in the plain search space (Sec. 4.3)."""
    S = [3, 2, 4, 3, 2]
    assert OF.profiling_space_size([S]) == int(np.prod(S)) == profiling_space_size([S])


def test_best_case_repeated_segment():
    """One distinct segment repeated, with the only cross-segment dependency from
    its last block to its first: product of the K strategy counts plus S_1 * S_K
    (Sec. 4.3; the product's index range is printed garbled and read as j = 1..K)."""
    S = [3, 4, 2, 5]
    want = int(np.prod(S)) + S[0] * S[-1]
    assert OF.profiling_space_size([S], [(0, 0, 3, 0)]) == want == profiling_space_size([S], [(0, 0, 3, 0)])


@pytest.mark.parametrize("seed", range(20))
def test_random_models_against_enumeration(seed):
    rs = np.random.default_rng([80, seed])
    n = int(rs.integers(1, 4))
    strategies = [[int(x) for x in rs.integers(1, 5, size=int(rs.integers(1, 5)))] for _ in range(n)]
    deps = []
    for _ in range(int(rs.integers(0, 5))):
        i, j = int(rs.integers(0, n)), int(rs.integers(0, n))
        deps.append((i, j, int(rs.integers(0, len(strategies[i]))), int(rs.integers(0, len(strategies[j])))))
    if deps and rs.random() < 0.3:
        deps.append(deps[0])  # a pair listed twice counts twice
    assert profiling_space_size(strategies, deps) == OF.profiling_space_size(strategies, deps)


def test_segment_plans_and_bad_inputs():
    assert segment_plans([3, 3, 3, 3]) == 81
    with pytest.raises(ValueError):
        profiling_space_size([])
    with pytest.raises(ValueError):
        profiling_space_size([[3, 0]])
    with pytest.raises(ValueError):
        profiling_space_size([[3, 3]], [(0, 1, 0, 0)])
    with pytest.raises(ValueError):
        profiling_space_size([[3, 3]], [(0, 0, 2, 0)])
