"""ctypes binding of the CPU oracle (liboracle.so, built from oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg.  The product package never imports it.

All arrays are host numpy arrays; results are int64 costs (INT64_MAX for an
infeasible search), int32 plans (-1 for an infeasible search) and int32
statuses (0 ok, 1 infeasible).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

INF64 = np.iinfo(np.int64).max
ST_OK = 0
ST_INFEASIBLE = 1


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc -O2 (plain loops, no vector intrinsics)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-pthread", SRC, "-o", tmp])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i = ctypes.c_int
        L.oracle_chain.argtypes = [i, i, i, i, P, P, P, P, P, P, i]
        L.oracle_chain.restype = i
        L.oracle_chain_mem.argtypes = [i, i, i, i, P, P, P, P, P, P, P, P, i]
        L.oracle_chain_mem.restype = i
        L.oracle_mem_frontier.argtypes = [i, i, i, i, P, P, P, P, i, P, i]
        L.oracle_mem_frontier.restype = i
        L.oracle_chain_values.argtypes = [i, i, i, P, P, P, P]
        L.oracle_chain_values.restype = i
        L.oracle_plan_cost.argtypes = [i, i, P, P, P, P]
        L.oracle_plan_cost.restype = ctypes.c_int64
        L.oracle_plan_mem.argtypes = [i, i, P, P]
        L.oracle_plan_mem.restype = ctypes.c_int64
        _lib = L
    return _lib


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def default_threads() -> int:
    return os.cpu_count() or 1


def chain(cost, rtab, redge, nthreads: int | None = None):
    """Unconstrained search.  cost [B][N][K] (or [N][K]), rtab [E][K][K],
    redge [N].  Returns (opt [B] int64, plan [B][N] int32, status [B] int32)."""
    cost = _c(cost, np.int32)
    single = cost.ndim == 2
    if single:
        cost = cost[None]
    B, N, K = cost.shape
    rtab = _c(rtab, np.int32)
    redge = _c(redge, np.int32)
    E = rtab.shape[0]
    assert rtab.shape == (E, K, K) and redge.shape == (N,)
    opt = np.empty(B, np.int64)
    plan = np.empty((B, N), np.int32)
    status = np.empty(B, np.int32)
    rc = lib().oracle_chain(N, K, B, E, _ptr(cost), _ptr(rtab), _ptr(redge), _ptr(opt), _ptr(plan),
                            _ptr(status), nthreads or default_threads())
    if rc != 0:
        raise ValueError("oracle_chain rejected its arguments")
    if single:
        return opt[0], plan[0], status[0]
    return opt, plan, status


def chain_mem(cost, rtab, redge, mem, budget, nthreads: int | None = None):
    """Memory-budgeted search; mem [B][N][K] uint8, budget [B] (inclusive)."""
    cost = _c(cost, np.int32)
    single = cost.ndim == 2
    if single:
        cost = cost[None]
        mem = np.asarray(mem)[None]
        budget = np.atleast_1d(budget)
    B, N, K = cost.shape
    rtab = _c(rtab, np.int32)
    redge = _c(redge, np.int32)
    mem = _c(mem, np.uint8)
    budget = _c(budget, np.int32)
    E = rtab.shape[0]
    assert mem.shape == (B, N, K) and budget.shape == (B,)
    opt = np.empty(B, np.int64)
    plan = np.empty((B, N), np.int32)
    status = np.empty(B, np.int32)
    rc = lib().oracle_chain_mem(N, K, B, E, _ptr(cost), _ptr(rtab), _ptr(redge), _ptr(mem), _ptr(budget),
                                _ptr(opt), _ptr(plan), _ptr(status), nthreads or default_threads())
    if rc != 0:
        raise ValueError("oracle_chain_mem rejected its arguments")
    if single:
        return opt[0], plan[0], status[0]
    return opt, plan, status


def mem_frontier(cost, rtab, redge, mem, n_mem: int, nthreads: int | None = None):
    """Budget frontier [B][n_mem] int64: entry m is the least cost of a plan
    whose memory total is at most m (INF64 where none fits)."""
    cost = _c(cost, np.int32)
    single = cost.ndim == 2
    if single:
        cost = cost[None]
        mem = np.asarray(mem)[None]
    B, N, K = cost.shape
    rtab = _c(rtab, np.int32)
    redge = _c(redge, np.int32)
    mem = _c(mem, np.uint8)
    E = rtab.shape[0]
    assert mem.shape == (B, N, K)
    out = np.empty((B, n_mem), np.int64)
    rc = lib().oracle_mem_frontier(N, K, B, E, _ptr(cost), _ptr(rtab), _ptr(redge), _ptr(mem), int(n_mem),
                                   _ptr(out), nthreads or default_threads())
    if rc != 0 or (out < 0).any():
        raise ValueError("oracle_mem_frontier rejected its arguments or ran out of memory")
    return out[0] if single else out


def expand_boundary(rbound, last, first):
    """Resharding tables of a segment chain written out plan by plan: the
    cost between plan t of one segment and plan s of the next is the boundary
    block pair's, R_e[t][s] = rbound[e][last[t]][first[s]] (Sec. 4.2: only
    the dependent block pairs at segment boundaries are profiled)."""
    rbound = np.asarray(rbound, np.int64)
    last = np.asarray(last, np.int64)
    first = np.asarray(first, np.int64)
    return np.ascontiguousarray(rbound[:, last[:, None], first[None, :]].astype(np.int32))


def segments(cost, rbound, last, first, redge, nthreads: int | None = None):
    """Segment-level search: the chain search of Eq. T over segments with the
    boundary-pair resharding tables expanded to K x K."""
    return chain(cost, expand_boundary(rbound, last, first), redge, nthreads=nthreads)


def chain_values(cost, rtab, redge):
    """Forward values D[i][s] (int64) of one chain, cost [N][K]."""
    cost = _c(cost, np.int32)
    N, K = cost.shape
    rtab = _c(rtab, np.int32)
    redge = _c(redge, np.int32)
    D = np.empty((N, K), np.int64)
    if lib().oracle_chain_values(N, K, rtab.shape[0], _ptr(cost), _ptr(rtab), _ptr(redge), _ptr(D)) != 0:
        raise ValueError("oracle_chain_values rejected its arguments")
    return D


def plan_cost(cost, rtab, redge, plan) -> int:
    """Eq. T of one plan of one chain (cost [N][K])."""
    cost = _c(cost, np.int32)
    N, K = cost.shape
    plan = _c(plan, np.int32)
    return int(lib().oracle_plan_cost(N, K, _ptr(cost), _ptr(_c(rtab, np.int32)), _ptr(_c(redge, np.int32)),
                                      _ptr(plan)))


def plan_mem(mem, plan) -> int:
    """Eq. M of one plan of one chain (mem [N][K])."""
    mem = _c(mem, np.uint8)
    N, K = mem.shape
    return int(lib().oracle_plan_mem(N, K, _ptr(mem), _ptr(_c(plan, np.int32))))
