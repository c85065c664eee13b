"""Brute-force enumeration of every plan of a tiny chain.

This is the pin for the oracle: it does not run the dynamic program at all.
It lists all S = prod_i D_i = K^N plans (Sec. 3.3: the search space is the
product of the per-block strategy counts), evaluates Eq. T (and Eq. M) of
Sec. 4.4 on each one directly, keeps the least, and breaks ties among the
optimal plans by taking the smallest in reversed lexicographic order
(x_{N-1}, x_{N-2}, ..., x_0) -- the closed characterisation of the
lowest-index-first traceback.
"""
from __future__ import annotations

import itertools

import numpy as np

COST_INF = 0x7FFFFFFF
INF64 = np.iinfo(np.int64).max


def all_plans(N: int, K: int) -> np.ndarray:
    """Every plan, shape [K^N, N]."""
    return np.array(list(itertools.product(range(K), repeat=N)), dtype=np.int64).reshape(-1, N)


def eq_T(cost: np.ndarray, rtab: np.ndarray, redge: np.ndarray, plans: np.ndarray) -> np.ndarray:
    """Eq. T for every row of `plans`; +inf (INF64) where a plan uses an
    unavailable strategy (cost 0x7FFFFFFF)."""
    N, K = cost.shape
    rows = np.arange(N)
    picked = cost[rows[None, :], plans]  # [P, N]
    bad = (picked == COST_INF).any(axis=1)
    total = picked.astype(np.int64).sum(axis=1)
    for i in range(1, N):
        total += rtab[redge[i], plans[:, i - 1], plans[:, i]].astype(np.int64)
    total[bad] = INF64
    return total


def eq_M(mem: np.ndarray, plans: np.ndarray) -> np.ndarray:
    N, K = mem.shape
    return mem[np.arange(N)[None, :], plans].astype(np.int64).sum(axis=1)


def solve(cost, rtab, redge, mem=None, budget=None):
    """(opt, plan, feasible) by enumeration; plan follows the reverse-lex rule."""
    cost = np.asarray(cost)
    N, K = cost.shape
    plans = all_plans(N, K)
    T = eq_T(cost, np.asarray(rtab), np.asarray(redge), plans)
    if mem is not None:
        T = T.copy()
        T[eq_M(np.asarray(mem), plans) > budget] = INF64
    best = T.min()
    if best == INF64:
        return INF64, np.full(N, -1, np.int64), False
    opt_plans = plans[T == best]
    # np.lexsort: the LAST key is primary -> keys x_0 .. x_{N-1} make x_{N-1} primary.
    order = np.lexsort([opt_plans[:, i] for i in range(N)])
    return int(best), opt_plans[order[0]], True
