"""Planted mistakes in the oracle must be caught by its pins.

Each case copies oracle.c, applies one plausible slip (a transposed operand,
a dropped term, a wrong index, a flipped tie-break, a wrong memory shift),
compiles the copy on the CPU, and checks that the brute-force / Dijkstra pins
reject it.  The real oracle is never modified.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np
import pytest

from oracle import oracle as O
from tests import brute
from tests.test_oracle_pins import dijkstra_cost, rand_chain

MUTANTS = {
    "transposed_R_forward": (
        "int64_t v = add_inf(prev[t], (int64_t)R[(size_t)t * K + s]);",
        "int64_t v = add_inf(prev[t], (int64_t)R[(size_t)s * K + t]);"),
    "dropped_block_cost": (
        "cur[s] = add_inf(best, cost_value(c[(size_t)i * K + s]));",
        "cur[s] = best;"),
    "dropped_first_block": (
        "for (int s = 0; s < K; ++s) D[s] = cost_value(c[s]);",
        "for (int s = 0; s < K; ++s) D[s] = 0;"),
    "edge_table_off_by_one": (
        "const int64_t *prev = D + (size_t)(i - 1) * K;\n    int64_t *cur",
        "const int64_t *prev = D + (size_t)(i - 1) * K; R = rtab + (size_t)redge[i - 1] * K * K;\n    int64_t *cur"),
    "final_tie_takes_last": (
        "if (last[s] < best) { best = last[s]; arg = s; }",
        "if (last[s] <= best) { best = last[s]; arg = s; }"),
    "traceback_tie_takes_last": (
        "if (add_inf(prev[t], (int64_t)R[(size_t)t * K + s]) == target) { pick = t; break; }",
        "if (add_inf(prev[t], (int64_t)R[(size_t)t * K + s]) == target) { pick = t; }"),
    "mem_shift_ignored": (
        "int64_t v = add_inf(D[DIDX(i - 1, t, m - ms)], (int64_t)R[(size_t)t * K + s]);",
        "int64_t v = add_inf(D[DIDX(i - 1, t, m)], (int64_t)R[(size_t)t * K + s]);"),
    "plan_mem_drops_block0": (
        "for (int i = 0; i < N; ++i) m += mem[(size_t)i * K + plan[i]];",
        "for (int i = 1; i < N; ++i) m += mem[(size_t)i * K + plan[i]];"),
    "plan_cost_drops_first_edge": (
        "for (int i = 1; i < N; ++i) {\n    const int32_t *R = rtab + (size_t)redge[i] * K * K;\n    t = add_inf",
        "for (int i = 2; i < N; ++i) {\n    const int32_t *R = rtab + (size_t)redge[i] * K * K;\n    t = add_inf"),
    "plan_cost_transposed_R": (
        "t = add_inf(t, (int64_t)R[(size_t)plan[i - 1] * K + plan[i]]);",
        "t = add_inf(t, (int64_t)R[(size_t)plan[i] * K + plan[i - 1]]);"),
    "mem_budget_exclusive": (
        "D[DIDX(0, s, m)] = (mem[s] <= m) ? cost_value(c[s]) : ORC_INF;",
        "D[DIDX(0, s, m)] = (mem[s] < m) ? cost_value(c[s]) : ORC_INF;"),
}


def build_mutant(tmp_path, name):
    src = open(O.SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"lib{name}.so"
    subprocess.check_call(["gcc", "-O1", "-shared", "-fPIC", "-pthread", str(path), "-o", str(so)])
    return str(so)


def pins_pass() -> bool:
    """A compact battery of the oracle's pins; False as soon as one fails."""
    rs = np.random.default_rng(99)
    for N, K in [(1, 3), (2, 2), (3, 3), (4, 2), (5, 3), (4, 4)]:
        for vals in [(0, 3), (0, 100)]:
            for _ in range(3):
                cost, rtab, redge = rand_chain(rs, N, K, 3, *vals)
                opt, plan, st = O.chain(cost, rtab, redge)
                bopt, bplan, _ = brute.solve(cost, rtab, redge)
                if opt != bopt or not np.array_equal(plan, bplan):
                    return False
                mem = rs.integers(0, 4, size=(N, K)).astype(np.uint8)
                budget = int(mem.min(axis=1).sum()) + 1
                opt, plan, st = O.chain_mem(cost, rtab, redge, mem, budget)
                bopt, bplan, ok = brute.solve(cost, rtab, redge, mem, budget)
                if (st == 0) != ok or (ok and (opt != bopt or not np.array_equal(plan, bplan))):
                    return False
    # the plan evaluators against Eq. T / Eq. M summed by the enumeration helpers
    for N, K in [(1, 3), (4, 3), (9, 5)]:
        cost, rtab, redge = rand_chain(rs, N, K, 3, 0, 1000)
        mem = rs.integers(0, 9, size=(N, K)).astype(np.uint8)
        plans = rs.integers(0, K, size=(8, N)).astype(np.int64)
        T, Mm = brute.eq_T(cost, rtab, redge, plans), brute.eq_M(mem, plans)
        for p, t, m in zip(plans, T, Mm):
            if O.plan_cost(cost, rtab, redge, p) != t or O.plan_mem(mem, p) != m:
                return False
    cost, rtab, redge = rand_chain(rs, 30, 8, 4, 10_000, 10**6)
    opt, _, _ = O.chain(cost, rtab, redge)
    return opt == dijkstra_cost(cost, rtab, redge)


def test_real_oracle_passes_battery():
    assert pins_pass()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name, monkeypatch):
    so = build_mutant(tmp_path, name)
    real = O.lib()
    L = ctypes.CDLL(so)
    for fn in ("oracle_chain", "oracle_chain_mem", "oracle_chain_values", "oracle_plan_cost", "oracle_plan_mem"):
        getattr(L, fn).argtypes = getattr(real, fn).argtypes
        getattr(L, fn).restype = getattr(real, fn).restype
    monkeypatch.setattr(O, "_lib", L)
    assert not pins_pass(), f"planted mistake {name} went unnoticed"
