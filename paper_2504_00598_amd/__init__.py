"""MI355X (gfx950) min-plus chain search: the plan-search dynamic program of
CFP (arXiv 2504.00598, Sec. 4.4) behind the C ABI of include/cfp.h.

    from paper_2504_00598_amd import search
    res = search.dp_chain(cost, rtab, redge)        # cost/rtab: int32 torch tensors on the GPU
    res.opt, res.status, res.plan
"""
from . import _lib  # noqa: F401
from ._lib import (CFP_COST_INF, CFP_ST_BADINPUT, CFP_ST_INFEASIBLE, CFP_ST_OK, CFP_V_CHAIN, CFP_V_MEM,  # noqa: F401
                   CFP_V_SCAN, CFP_V_SEG, CfpError, Desc, SegDesc, cfp_dp_chain, cfp_dp_chain_mem, cfp_dp_segments,
                   cfp_mem_frontier, cfp_minplus_scan, cfp_traceback_segments,
                   cfp_r_limit,
                   cfp_traceback, cfp_workspace_bytes, status_string)
