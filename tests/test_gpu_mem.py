"""GPU parity of cfp_dp_chain_mem + cfp_traceback against the CPU oracle:
optimum, status and plan must match bit for bit."""
from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_util import assert_mem_parity, need_gpu, run_mem, say
from workloads import configs, gen

pytestmark = pytest.mark.gpu
INF = gen.COST_INF


def mem_case(seed, B, N, K, E, lo, hi, mlo, mhi, M):
    rs = np.random.default_rng(seed)
    cost = rs.integers(lo, hi, size=(B, N, K)).astype(np.int32)
    rtab = rs.integers(lo, hi, size=(E, K, K)).astype(np.int32)
    rtab[:, np.arange(K), np.arange(K)] = 0
    redge = (np.arange(N) % E).astype(np.int32)
    mem = rs.integers(mlo, mhi, size=(B, N, K)).astype(np.uint8)
    return cost, rtab, redge, mem


def test_config_full():
    need_gpu()
    say("config mem_llama_n288_k32")
    d = configs.make("mem_llama_n288_k32")
    assert_mem_parity(d["cost"], d["rtab"], d["redge"], d["mem"], d["M"], d["budget"], "mem config")


@pytest.mark.parametrize("N,K,M", [(1, 5, 10), (2, 3, 7), (13, 16, 64), (40, 32, 65), (70, 20, 130), (25, 32, 200),
                                   (90, 9, 300)])
def test_shapes(N, K, M):
    need_gpu()
    say("mem shape", N, K, M)
    cost, rtab, redge, mem = mem_case([N, K, M], 6, N, K, 12, 10_000, 1_000_000, 0, min(9, M), M)  # entries < M
    lo = mem.min(axis=2).sum(axis=1)
    hi = mem.max(axis=2).sum(axis=1)
    # budgets spanning infeasible, tight, middle, loose and the top bucket
    budget = np.array([max(int(lo[0]) - 1, 0), int(lo[1]), (int(lo[2]) + int(hi[2])) // 2, int(hi[3]), M - 1,
                       min(M - 1, int(lo[5]) + 3)], np.int32)
    budget = np.minimum(budget, M - 1)
    assert_mem_parity(cost, rtab, redge, mem, M, budget, f"N={N} K={K} M={M}")


@pytest.mark.parametrize("K", [4, 32])
def test_heavy_ties(K):
    need_gpu()
    N, M = 30, 100
    cost, rtab, redge, mem = mem_case([7, K], 4, N, K, 3, 0, 3, 0, 3, M)
    budget = np.array([10, 20, 40, 99], np.int32)
    assert_mem_parity(cost, rtab, redge, mem, M, budget, f"ties K={K}")


def test_large_shifts_and_general_edges():
    need_gpu()
    rs = np.random.default_rng(11)
    B, N, K, E, M = 3, 50, 12, 5, 700
    cost = rs.integers(0, 10**6, size=(B, N, K)).astype(np.int32)
    rtab = rs.integers(0, 10**6, size=(E, K, K)).astype(np.int32)
    redge = rs.integers(0, E, size=N).astype(np.int32)
    mem = rs.integers(0, 17, size=(B, N, K)).astype(np.uint8)   # shifts up to the supported 16
    budget = np.array([699, 300, 150], np.int32)
    assert_mem_parity(cost, rtab, redge, mem, M, budget, "shift16")


def test_unavailable_and_statuses():
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT, CFP_ST_INFEASIBLE
    cost, rtab, redge, mem = mem_case(12, 4, 20, 8, 2, 0, 100, 0, 5, 64)
    cost[0][cost[0] % 3 == 0] = INF
    cost[1, 5, :] = INF                         # infeasible
    mem[2, 3, 2] = 40                           # beyond the largest supported shift -> bad input
    budget = np.array([63, 63, 63, 2], np.int32)  # search 3: budget below the least memory plan
    opt, st, plan = run_mem(cost, rtab, redge, mem, 64, budget)
    assert st[1] == CFP_ST_INFEASIBLE and st[2] == CFP_ST_BADINPUT
    assert (plan[1] == -1).all() and (plan[2] == -1).all()
    good = [0, 3]
    assert_mem_parity(cost[good], rtab, redge, mem[good], 64, budget[good], "inf")


def test_budget_out_of_range_is_bad_input():
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT
    cost, rtab, redge, mem = mem_case(13, 2, 10, 4, 2, 0, 100, 0, 3, 32)
    opt, st, plan = run_mem(cost, rtab, redge, mem, 32, np.array([31, 32], np.int32))
    assert st[0] == 0 and st[1] == CFP_ST_BADINPUT


@pytest.mark.parametrize("bad", ["limit", "negative"])
def test_resharding_out_of_range_is_bad_input(bad):
    """The memory forward checks the range of R while packing it."""
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT, cfp_r_limit
    cost, rtab, redge, mem = mem_case(14, 3, 30, 32, 3, 0, 100, 0, 4, 64)
    rtab[2, 31, 5] = cfp_r_limit(1, 32) if bad == "limit" else -1
    opt, st, plan = run_mem(cost, rtab, redge, mem, 64, np.array([63, 40, 20], np.int32))
    assert (st == CFP_ST_BADINPUT).all() and (plan == -1).all()


def test_periodic_layers():
    """Repeated layers (the same costs and memory every 12 blocks): many tied
    plans at every budget."""
    need_gpu()
    rs = np.random.default_rng(31)
    B, N, K, M = 4, 96, 32, 300
    cost = np.tile(rs.integers(0, 40, size=(B, 12, K)).astype(np.int32), (1, N // 12, 1))
    mem = np.tile(rs.integers(0, 5, size=(B, 12, K)).astype(np.uint8), (1, N // 12, 1))
    rtab = rs.integers(0, 40, size=(12, K, K)).astype(np.int32)
    redge = (np.arange(N) % 12).astype(np.int32)
    budget = np.array([60, 120, 200, 299], np.int32)
    assert_mem_parity(cost, rtab, redge, mem, M, budget, "periodic")
