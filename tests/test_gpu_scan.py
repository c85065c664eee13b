"""GPU parity of cfp_minplus_scan + cfp_traceback against the CPU oracle's
sequential dynamic program: the tree of min-plus products must reach the same
optimum and the same lowest-index plan, bit for bit."""
from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_util import assert_scan_parity, need_gpu, run_scan, say
from workloads import configs, gen

pytestmark = pytest.mark.gpu
INF = gen.COST_INF


def case(seed, B, N, K, E, lo, hi):
    rs = np.random.default_rng(seed)
    cost = rs.integers(lo, hi, size=(B, N, K)).astype(np.int32)
    rtab = rs.integers(lo, hi, size=(E, K, K)).astype(np.int32)
    redge = rs.integers(0, E, size=N).astype(np.int32)
    return cost, rtab, redge


# odd and even chain lengths (unpaired nodes carried up), padded and full K
SHAPES = [(1, 5), (2, 3), (3, 16), (5, 100), (6, 128), (7, 129), (33, 130), (20, 256), (9, 512), (64, 64),
          (100, 31)]


@pytest.mark.parametrize("N,K", SHAPES)
def test_shapes(N, K):
    need_gpu()
    say("scan shape", N, K)
    from paper_2504_00598_amd import cfp_r_limit
    rhi = min(1_000_000, cfp_r_limit(2, K))
    cost, rtab, redge = case([N, K], 3, N, K, 4, 10_000, 1_000_000)
    rtab = np.minimum(rtab, rhi - 1).astype(np.int32)
    assert_scan_parity(cost, rtab, redge, f"N={N} K={K}")


@pytest.mark.parametrize("N,K", [(9, 3), (40, 16), (13, 128), (6, 200)])
def test_heavy_ties(N, K):
    need_gpu()
    cost, rtab, redge = case([5, N, K], 2, N, K, 3, 0, 3)
    assert_scan_parity(cost, rtab, redge, f"ties N={N} K={K}")


def test_unavailable_and_infeasible():
    need_gpu()
    cost, rtab, redge = case(6, 3, 25, 40, 2, 0, 1000)
    rs = np.random.default_rng(7)
    cost[0][rs.random((25, 40)) < 0.3] = INF
    cost[1, 11, :] = INF
    assert_scan_parity(cost, rtab, redge, "inf")


def test_cost_spread_beyond_range_is_bad_input():
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT
    cost, rtab, redge = case(8, 2, 10, 8, 2, 0, 100)
    cost[1, 4, 3] = 2 ** 30 + 1000   # finite costs of one block more than 2^30 apart
    opt, st, plan = run_scan(cost, rtab, redge)
    assert st.tolist() == [0, CFP_ST_BADINPUT] and (plan[1] == -1).all()


def test_config_full():
    need_gpu()
    say("config scan_n4096_k512")
    d = configs.make("scan_n4096_k512")
    assert_scan_parity(d["cost"], d["rtab"], d["redge"], "scan config")


def test_repeat_is_bit_identical():
    """The product tree, down-sweep and traceback give the same optimum, status
    and plan on every call (a fresh workspace each time), and the first call
    matches the oracle."""
    need_gpu()
    say("scan repeat")
    d = configs.make("scan_n4096_k512")
    cost = np.ascontiguousarray(d["cost"][:2, :300])
    redge = np.ascontiguousarray(d["redge"][:300])
    assert_scan_parity(cost, d["rtab"], redge, "scan repeat, first call")
    a = run_scan(cost, d["rtab"], redge)
    for _ in range(3):
        b = run_scan(cost, d["rtab"], redge)
        for x, y in zip(a, b):
            np.testing.assert_array_equal(x, y)
