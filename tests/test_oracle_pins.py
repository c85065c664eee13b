"""Pins of the CPU oracle against facts that do not come from the oracle.

  - brute-force enumeration of every plan (Eq. T / Eq. M evaluated directly),
    including the reverse-lexicographic tie rule;
  - hand-worked fixtures under tests/golden/;
  - closed forms: R == 0, K == 1, N == 1, memory thresholds;
  - a library routine: Dijkstra on the layered DAG (scipy);
  - invariants: Eq. T of the returned plan equals the optimum, shift and
    reversal invariance, monotonicity in the budget.
"""
from __future__ import annotations

import glob
import json
import os

import numpy as np
import pytest

from oracle import oracle as O
from tests import brute
from workloads import gen

HERE = os.path.dirname(os.path.abspath(__file__))
rng_seed = 20240401


def rand_chain(rs, N, K, E, lo, hi, inf_frac=0.0):
    cost = rs.integers(lo, hi, size=(N, K)).astype(np.int32)
    if inf_frac:
        cost[rs.random((N, K)) < inf_frac] = brute.COST_INF
    rtab = rs.integers(lo, hi, size=(E, K, K)).astype(np.int32)
    redge = rs.integers(0, E, size=N).astype(np.int32)
    return cost, rtab, redge


def eval_T(cost, rtab, redge, plan):
    return int(brute.eq_T(cost, rtab, redge, np.asarray(plan, np.int64)[None])[0])


# ----------------------------------------------------------- brute force --

TINY = [(N, K) for N in range(1, 6) for K in range(1, 5)]


@pytest.mark.parametrize("N,K", TINY)
@pytest.mark.parametrize("vals", [(0, 3), (0, 50), (10_000, 1_000_000)])
def test_chain_vs_brute_tiny(N, K, vals):
    rs = np.random.default_rng([rng_seed, N, K, vals[1]])
    for rep in range(4):
        cost, rtab, redge = rand_chain(rs, N, K, 3, *vals)
        opt, plan, st = O.chain(cost, rtab, redge)
        bopt, bplan, ok = brute.solve(cost, rtab, redge)
        assert ok and st == O.ST_OK
        assert opt == bopt
        np.testing.assert_array_equal(plan, bplan)


def test_chain_vs_brute_random_shapes():
    rs = np.random.default_rng(rng_seed + 1)
    done = 0
    while done < 40:
        N = int(rs.integers(2, 12))
        K = int(rs.integers(2, 9))
        if K ** N > 65536:
            continue
        lo, hi = [(0, 3), (0, 1000), (10_000, 10_000_000)][done % 3]
        cost, rtab, redge = rand_chain(rs, N, K, int(rs.integers(1, 5)), lo, hi)
        opt, plan, st = O.chain(cost, rtab, redge)
        bopt, bplan, _ = brute.solve(cost, rtab, redge)
        assert opt == bopt
        np.testing.assert_array_equal(plan, bplan)
        done += 1


def test_chain_unavailable_strategies_vs_brute():
    rs = np.random.default_rng(rng_seed + 2)
    for rep in range(60):
        N, K = int(rs.integers(1, 6)), int(rs.integers(1, 5))
        cost, rtab, redge = rand_chain(rs, N, K, 2, 0, 20, inf_frac=0.35)
        opt, plan, st = O.chain(cost, rtab, redge)
        bopt, bplan, ok = brute.solve(cost, rtab, redge)
        if ok:
            assert st == O.ST_OK and opt == bopt
            np.testing.assert_array_equal(plan, bplan)
        else:
            assert st == O.ST_INFEASIBLE and opt == O.INF64
            assert (plan == -1).all()


@pytest.mark.parametrize("N,K", [(n, k) for n in range(1, 6) for k in range(1, 5)])
def test_mem_vs_brute_tiny(N, K):
    rs = np.random.default_rng([rng_seed + 3, N, K])
    for rep in range(3):
        cost, rtab, redge = rand_chain(rs, N, K, 2, 0, 4)
        mem = rs.integers(0, 4, size=(N, K)).astype(np.uint8)
        lo = int(mem.min(axis=1).sum())
        hi = int(mem.max(axis=1).sum())
        for budget in sorted({0, max(lo - 1, 0), lo, (lo + hi) // 2, hi, hi + 2}):
            opt, plan, st = O.chain_mem(cost, rtab, redge, mem, budget)
            bopt, bplan, ok = brute.solve(cost, rtab, redge, mem, budget)
            if ok:
                assert st == O.ST_OK and opt == bopt, (budget, opt, bopt)
                np.testing.assert_array_equal(plan, bplan)
            else:
                assert st == O.ST_INFEASIBLE and (plan == -1).all()


def test_mem_vs_brute_random_shapes():
    rs = np.random.default_rng(rng_seed + 4)
    done = 0
    while done < 30:
        N = int(rs.integers(2, 10))
        K = int(rs.integers(2, 7))
        if K ** N > 65536:
            continue
        cost, rtab, redge = rand_chain(rs, N, K, 3, 0, 1000)
        mem = rs.integers(0, 9, size=(N, K)).astype(np.uint8)
        budget = int(rs.integers(int(mem.min(axis=1).sum()), int(mem.max(axis=1).sum()) + 1))
        opt, plan, st = O.chain_mem(cost, rtab, redge, mem, budget)
        bopt, bplan, ok = brute.solve(cost, rtab, redge, mem, budget)
        assert ok and opt == bopt
        np.testing.assert_array_equal(plan, bplan)
        done += 1


# --------------------------------------------------------------- golden --

def _load(name):
    with open(os.path.join(HERE, "golden", name)) as f:
        return json.load(f)


@pytest.mark.parametrize("name", ["chain_n3_k2.json", "chain_ties_n3_k2.json"])
def test_golden_chain(name):
    g = _load(name)
    opt, plan, st = O.chain(np.array(g["cost"]), np.array(g["rtab"]), np.array(g["redge"]))
    assert st == 0 and opt == g["opt"]
    assert plan.tolist() == g["plan"]


def test_golden_mem():
    g = _load("mem_n3_k2.json")
    for case in g["cases"]:
        opt, plan, st = O.chain_mem(np.array(g["cost"]), np.array(g["rtab"]), np.array(g["redge"]),
                                    np.array(g["mem"]), case["budget"])
        if case["feasible"]:
            assert st == 0 and opt == case["opt"]
        else:
            assert st == O.ST_INFEASIBLE
        assert plan.tolist() == case["plan"]


def test_golden_files_cite_the_paper():
    for path in glob.glob(os.path.join(HERE, "golden", "*.json")):
        with open(path) as f:
            assert "Sec." in json.load(f)["cite"], path


# ----------------------------------------------------------- closed forms --

@pytest.mark.parametrize("N,K", [(1, 7), (5, 3), (40, 16), (300, 64)])
def test_zero_resharding_is_sum_of_block_minima(N, K):
    rs = np.random.default_rng([rng_seed + 5, N, K])
    cost = rs.integers(0, 1000, size=(N, K)).astype(np.int32)
    rtab = np.zeros((3, K, K), np.int32)
    redge = rs.integers(0, 3, size=N).astype(np.int32)
    opt, plan, st = O.chain(cost, rtab, redge)
    assert opt == int(cost.min(axis=1).astype(np.int64).sum())
    np.testing.assert_array_equal(plan, cost.argmin(axis=1))  # argmin picks the lowest index


def test_single_strategy_closed_form():
    rs = np.random.default_rng(rng_seed + 6)
    N = 50
    cost = rs.integers(0, 10**7, size=(N, 1)).astype(np.int32)
    rtab = rs.integers(0, 10**7, size=(4, 1, 1)).astype(np.int32)
    redge = rs.integers(0, 4, size=N).astype(np.int32)
    opt, plan, st = O.chain(cost, rtab, redge)
    want = int(cost[:, 0].astype(np.int64).sum()) + sum(int(rtab[redge[i], 0, 0]) for i in range(1, N))
    assert opt == want and (plan == 0).all()


def test_single_block_closed_form():
    cost = np.array([[7, 3, 9, 3]], np.int32)
    opt, plan, st = O.chain(cost, np.zeros((1, 4, 4), np.int32), np.zeros(1, np.int32))
    assert opt == 3 and plan.tolist() == [1]


# ---------------------------------------------------------- library pin --

def dijkstra_cost(cost, rtab, redge):
    """Least source-to-sink distance on the layered DAG with scipy's Dijkstra.
    Every edge weight is shifted by +1 (csgraph drops explicit zeros); every
    source-to-sink path has exactly N+1 edges, so the shift is N+1."""
    from scipy.sparse import csr_matrix
    from scipy.sparse.csgraph import shortest_path

    N, K = cost.shape
    src, sink = N * K, N * K + 1
    rows, cols, w = [], [], []
    for s in range(K):
        rows.append(src); cols.append(s); w.append(float(cost[0, s]) + 1)
    for i in range(1, N):
        R = rtab[redge[i]].astype(np.float64)
        t_idx, s_idx = np.meshgrid(np.arange(K), np.arange(K), indexing="ij")
        rows.extend(((i - 1) * K + t_idx).ravel().tolist())
        cols.extend((i * K + s_idx).ravel().tolist())
        w.extend((R + cost[i][None, :].astype(np.float64) + 1).ravel().tolist())
    for s in range(K):
        rows.append((N - 1) * K + s); cols.append(sink); w.append(1.0)
    G = csr_matrix((w, (rows, cols)), shape=(N * K + 2, N * K + 2))
    d = shortest_path(G, method="D", directed=True, indices=[src])[0, sink]
    return int(round(d)) - (N + 1)


@pytest.mark.parametrize("N,K,seed", [(2, 3, 0), (17, 8, 1), (60, 24, 2), (200, 64, 3)])
def test_cost_equals_dijkstra(N, K, seed):
    rs = np.random.default_rng([rng_seed + 7, seed])
    cost, rtab, redge = rand_chain(rs, N, K, 5, 10_000, 10_000_000)
    opt, plan, st = O.chain(cost, rtab, redge)
    assert opt == dijkstra_cost(cost, rtab, redge)


# ------------------------------------------------------------ invariants --

@pytest.mark.parametrize("N,K", [(30, 16), (200, 64), (64, 128)])
def test_plan_cost_equals_opt(N, K):
    rs = np.random.default_rng([rng_seed + 8, N, K])
    cost, rtab, redge = rand_chain(rs, N, K, 12, 10_000, 10_000_000)
    opt, plan, st = O.chain(cost, rtab, redge)
    assert eval_T(cost, rtab, redge, plan) == opt
    assert O.plan_cost(cost, rtab, redge, plan) == opt


@pytest.mark.parametrize("N,K,E", [(1, 1, 1), (1, 5, 2), (2, 3, 1), (7, 4, 3), (40, 9, 5), (300, 33, 12)])
def test_plan_evaluators_vs_direct_sums(N, K, E):
    """oracle_plan_cost and oracle_plan_mem on arbitrary plans (not only the
    optimal one) equal Eq. T and Eq. M summed directly by the enumeration
    helpers: every block's cost and memory, every edge's table entry, and
    +inf for a plan through an unavailable strategy."""
    rs = np.random.default_rng([rng_seed + 30, N, K, E])
    cost, rtab, redge = rand_chain(rs, N, K, E, 0, 2**31 - 1, inf_frac=0.05)
    mem = rs.integers(0, 256, size=(N, K)).astype(np.uint8)
    plans = rs.integers(0, K, size=(50, N)).astype(np.int64)
    T = brute.eq_T(cost, rtab, redge, plans)
    Mm = brute.eq_M(mem, plans)
    for p, t, m in zip(plans, T, Mm):
        assert O.plan_cost(cost, rtab, redge, p) == t
        assert O.plan_mem(mem, p) == m
    # a hand-summed case: block 0 alone carries all the memory and the cost
    cost1 = np.zeros((N, K), np.int32)
    cost1[0, :] = 7
    mem1 = np.zeros((N, K), np.uint8)
    mem1[0, :] = 3
    z = np.zeros((E, K, K), np.int32)
    p0 = np.zeros(N, np.int64)
    assert O.plan_cost(cost1, z, redge, p0) == 7
    assert O.plan_mem(mem1, p0) == 3


def test_shift_invariance():
    rs = np.random.default_rng(rng_seed + 9)
    N, K, E = 60, 12, 4
    cost, rtab, redge = rand_chain(rs, N, K, E, 0, 1000)
    opt, plan, _ = O.chain(cost, rtab, redge)
    # add delta to one block's cost row: opt moves by delta, plan unchanged
    c2 = cost.copy(); c2[17] += 555
    opt2, plan2, _ = O.chain(c2, rtab, redge)
    assert opt2 == opt + 555
    np.testing.assert_array_equal(plan2, plan)
    # add delta to every entry of one table: opt moves by (#edges using it) * delta
    e = int(redge[5])
    uses = int((redge[1:] == e).sum())
    r2 = rtab.copy(); r2[e] += 77
    opt3, plan3, _ = O.chain(cost, r2, redge)
    assert opt3 == opt + uses * 77
    np.testing.assert_array_equal(plan3, plan)


def test_reversal_invariance():
    rs = np.random.default_rng(rng_seed + 10)
    for rep in range(5):
        N, K, E = 40, 9, 3
        cost, rtab, redge = rand_chain(rs, N, K, E, 0, 10**6)
        opt, _, _ = O.chain(cost, rtab, redge)
        # reversed chain: block i' = N-1-i; edge into i' uses the transposed table of original edge N-i'
        rc = cost[::-1].copy()
        rt = np.ascontiguousarray(np.transpose(rtab, (0, 2, 1)))
        re = np.zeros(N, np.int32)
        re[1:] = redge[N - np.arange(1, N)]
        opt_r, _, _ = O.chain(rc, rt, re)
        assert opt_r == opt


def test_mem_unconstrained_cases_match_chain():
    rs = np.random.default_rng(rng_seed + 11)
    N, K = 40, 8
    cost, rtab, redge = rand_chain(rs, N, K, 3, 0, 10**6)
    opt, plan, _ = O.chain(cost, rtab, redge)
    zero = np.zeros((N, K), np.uint8)
    o1, p1, s1 = O.chain_mem(cost, rtab, redge, zero, 0)
    assert s1 == 0 and o1 == opt
    np.testing.assert_array_equal(p1, plan)
    mem = rs.integers(0, 9, size=(N, K)).astype(np.uint8)
    big = int(mem.max(axis=1).sum())
    o2, p2, s2 = O.chain_mem(cost, rtab, redge, mem, big)
    assert s2 == 0 and o2 == opt
    np.testing.assert_array_equal(p2, plan)


def test_mem_feasibility_threshold_and_monotone():
    rs = np.random.default_rng(rng_seed + 12)
    N, K = 30, 6
    cost, rtab, redge = rand_chain(rs, N, K, 3, 0, 10**5)
    mem = rs.integers(0, 9, size=(N, K)).astype(np.uint8)
    lo = int(mem.min(axis=1).sum())
    _, p, st = O.chain_mem(cost, rtab, redge, mem, lo - 1)
    assert st == O.ST_INFEASIBLE and (p == -1).all()
    prev = None
    for budget in range(lo, int(mem.max(axis=1).sum()) + 1, 3):
        o, p, st = O.chain_mem(cost, rtab, redge, mem, budget)
        assert st == 0
        assert O.plan_mem(mem, p) <= budget
        assert eval_T(cost, rtab, redge, p) == o
        if prev is not None:
            assert o <= prev
        prev = o


def test_batched_equals_single():
    rs = np.random.default_rng(rng_seed + 13)
    B, N, K = 5, 20, 7
    cost = rs.integers(0, 100, size=(B, N, K)).astype(np.int32)
    rtab = rs.integers(0, 100, size=(2, K, K)).astype(np.int32)
    redge = rs.integers(0, 2, size=N).astype(np.int32)
    opt, plan, st = O.chain(cost, rtab, redge, nthreads=3)
    for b in range(B):
        o, p, s = O.chain(cost[b], rtab, redge, nthreads=1)
        assert o == opt[b]
        np.testing.assert_array_equal(p, plan[b])


def test_chain_values_last_row_min_is_opt():
    rs = np.random.default_rng(rng_seed + 14)
    cost, rtab, redge = rand_chain(rs, 25, 6, 2, 0, 1000)
    D = O.chain_values(cost, rtab, redge)
    opt, _, _ = O.chain(cost, rtab, redge)
    assert D[-1].min() == opt
    assert (D[0] == cost[0]).all()


# ------------------------------------------------ budget frontier (f2) ----

@pytest.mark.parametrize("N,K", [(1, 3), (2, 2), (3, 3), (4, 3), (5, 2)])
def test_mem_frontier_vs_brute(N, K):
    """Every entry of the frontier is the least Eq. T cost over the plans
    whose Eq. M total is at most m (Sec. 4.4), enumerated directly."""
    rs = np.random.default_rng(rng_seed + 40 + N * 7 + K)
    for trial in range(4):
        vals = 3 if trial % 2 else 50
        cost = rs.integers(0, vals, size=(N, K)).astype(np.int32)
        if trial == 3:
            cost[rs.integers(0, N), rs.integers(0, K)] = brute.COST_INF
        rtab = rs.integers(0, vals, size=(2, K, K)).astype(np.int32)
        redge = rs.integers(0, 2, size=N).astype(np.int32)
        mem = rs.integers(0, 4, size=(N, K)).astype(np.uint8)
        M = int(mem.max(axis=1).sum()) + 2
        F = O.mem_frontier(cost, rtab, redge, mem, M)
        plans = brute.all_plans(N, K)
        T = brute.eq_T(cost, rtab, redge, plans)
        Mp = brute.eq_M(mem, plans)
        for m in range(M):
            fit = T[Mp <= m]
            want = int(fit.min()) if fit.size else brute.INF64
            assert F[m] == want, (trial, m)


def test_mem_frontier_matches_single_budget_searches():
    rs = np.random.default_rng(rng_seed + 41)
    B, N, K = 3, 18, 5
    cost = rs.integers(0, 1000, size=(B, N, K)).astype(np.int32)
    rtab = rs.integers(0, 1000, size=(3, K, K)).astype(np.int32)
    redge = rs.integers(0, 3, size=N).astype(np.int32)
    mem = rs.integers(0, 6, size=(B, N, K)).astype(np.uint8)
    M = 70
    F = O.mem_frontier(cost, rtab, redge, mem, M)
    for b in range(B):
        prev = brute.INF64
        for m in range(M):
            o, p, st = O.chain_mem(cost[b], rtab, redge, mem[b], m)
            assert F[b, m] == o
            assert F[b, m] <= prev  # more memory never costs more
            prev = F[b, m]
        # with room for every plan the frontier ends at the unconstrained optimum
        if int(mem[b].max(axis=1).sum()) < M:
            assert F[b, -1] == O.chain(cost[b], rtab, redge)[0]


# ---------------------------------------- segments with boundary resharding ----

def seg_eq_T(cost, rbound, last, first, redge, plan):
    """Eq. T of one plan of a segment chain, from its definition: segment
    costs plus the boundary block pair's resharding at every boundary."""
    t = 0
    for i, x in enumerate(plan):
        if cost[i, x] == brute.COST_INF:
            return brute.INF64
        t += int(cost[i, x])
    for i in range(1, len(plan)):
        t += int(rbound[redge[i], last[plan[i - 1]], first[plan[i]]])
    return t


def digit_maps(P, S):
    """Plan t = sum_j x_j S^j of P blocks with S strategies: first block x_0,
    last block x_{P-1} (the numbering used for segments of P blocks)."""
    t = np.arange(S ** P)
    return (t // S ** (P - 1)).astype(np.uint8), (t % S).astype(np.uint8)


@pytest.mark.parametrize("N,P,S", [(1, 2, 2), (2, 2, 2), (3, 2, 2), (4, 2, 2), (3, 1, 3), (2, 3, 2)])
def test_segments_vs_brute(N, P, S):
    rs = np.random.default_rng(rng_seed + 60 + N * 10 + P * 3 + S)
    K = S ** P
    last, first = digit_maps(P, S)
    for trial in range(4):
        vals = 3 if trial % 2 else 100
        cost = rs.integers(0, vals, size=(N, K)).astype(np.int32)
        if trial == 3:
            cost[rs.integers(0, N), rs.integers(0, K)] = brute.COST_INF
        rbound = rs.integers(0, vals, size=(2, S, S)).astype(np.int32)
        redge = rs.integers(0, 2, size=N).astype(np.int32)
        opt, plan, st = O.segments(cost, rbound, last, first, redge)
        plans = brute.all_plans(N, K)
        T = np.array([seg_eq_T(cost, rbound, last, first, redge, p) for p in plans])
        best = T.min()
        assert opt == best
        assert seg_eq_T(cost, rbound, last, first, redge, plan) == opt
        ties = plans[T == best]
        order = np.lexsort([ties[:, i] for i in range(N)])
        np.testing.assert_array_equal(plan, ties[order[0]])  # lowest index at every choice


def test_segments_zero_boundary_is_sum_of_minima():
    rs = np.random.default_rng(rng_seed + 61)
    N, K = 12, 81
    last, first = digit_maps(4, 3)
    cost = rs.integers(0, 10**6, size=(N, K)).astype(np.int32)
    rbound = np.zeros((1, 3, 3), np.int32)
    opt, plan, st = O.segments(cost, rbound, last, first, np.zeros(N, np.int32))
    assert opt == int(cost.min(axis=1).sum())
    np.testing.assert_array_equal(plan, cost.argmin(axis=1))


def test_expand_boundary_layout():
    # R[t][s] takes the row from t's last block and the column from s's first block
    rb = np.arange(2 * 3 * 3, dtype=np.int32).reshape(2, 3, 3)
    last, first = digit_maps(2, 3)  # t = x0 + 3 x1: last = x1, first = x0
    R = O.expand_boundary(rb, last, first)
    for e in range(2):
        for t in range(9):
            for s in range(9):
                assert R[e, t, s] == rb[e, t // 3, s % 3]
