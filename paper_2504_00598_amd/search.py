"""Convenience calls: one forward variant followed by the traceback, on the
current stream.  Each returns device tensors (opt [B] int64, status [B]
int32, plan [B][N] int32) and the workspace."""
from __future__ import annotations

from dataclasses import dataclass

from . import _lib as L


@dataclass
class Result:
    opt: object
    status: object
    plan: object
    ws: object


def dp_chain(cost, rtab, redge, ws=None, stream=None) -> Result:
    d = L.Desc(cost, rtab, redge)
    opt, status, ws = L.cfp_dp_chain(d, ws=ws, stream=stream)
    plan = L.cfp_traceback(d, L.CFP_V_CHAIN, ws, stream=stream)
    return Result(opt, status, plan, ws)


def dp_chain_mem(cost, rtab, redge, mem, n_mem, budget, ws=None, stream=None) -> Result:
    d = L.Desc(cost, rtab, redge)
    opt, status, ws = L.cfp_dp_chain_mem(d, mem, n_mem, budget, ws=ws, stream=stream)
    plan = L.cfp_traceback(d, L.CFP_V_MEM, ws, n_mem=n_mem, stream=stream)
    return Result(opt, status, plan, ws)


def mem_frontier(cost, rtab, redge, mem, n_mem, ws=None, stream=None):
    """Least cost at every memory budget 0 .. n_mem-1 (frontier [B][n_mem]
    int64), the status of each search, and the plans at budget n_mem-1."""
    d = L.Desc(cost, rtab, redge)
    frontier, status, ws = L.cfp_mem_frontier(d, mem, n_mem, ws=ws, stream=stream)
    plan = L.cfp_traceback(d, L.CFP_V_MEM, ws, n_mem=n_mem, stream=stream)
    return frontier, status, plan, ws


def dp_segments(cost, rbound, last, first, redge, ws=None, stream=None) -> Result:
    """Segment-level search with boundary resharding: cost [B][N][K], rbound
    [E][L][F], last/first [K] (device tensors), redge [N] (host)."""
    d = L.SegDesc(cost, rbound, last, first, redge)
    opt, status, ws = L.cfp_dp_segments(d, ws=ws, stream=stream)
    plan = L.cfp_traceback_segments(d, ws, stream=stream)
    return Result(opt, status, plan, ws)


def minplus_scan(cost, rtab, redge, ws=None, stream=None) -> Result:
    d = L.Desc(cost, rtab, redge)
    opt, status, ws = L.cfp_minplus_scan(d, ws=ws, stream=stream)
    plan = L.cfp_traceback(d, L.CFP_V_SCAN, ws, stream=stream)
    return Result(opt, status, plan, ws)
