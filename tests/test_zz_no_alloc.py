"""cfp_search_chain_noalloc (the entry point for callers that cannot
allocate) against cfp_dp_chain + cfp_traceback on their own workspace: the
same optimum, status and plan, over two calls in a row whose second is
smaller, so that the second runs on the static scratch the first one left."""
from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_util import dev, need_gpu, say
from workloads import configs

pytestmark = pytest.mark.gpu


def _reference(cost, rtab, redge):
    import torch
    from paper_2504_00598_amd import search

    r = search.dp_chain(dev(cost), dev(rtab), redge)
    torch.cuda.synchronize()
    return r.opt.cpu().numpy(), r.status.cpu().numpy(), r.plan.cpu().numpy()


def _noalloc(cost, rtab, redge):
    import torch
    from paper_2504_00598_amd import _lib as L

    d = L.Desc(dev(cost), dev(rtab), redge)
    opt, status, plan = L.cfp_search_chain_noalloc(d)
    torch.cuda.synchronize()
    return opt.cpu().numpy(), status.cpu().numpy(), plan.cpu().numpy()


def test_noalloc_matches_workspace_calls():
    need_gpu()
    # first: the 1152-block K=64 chain with 64 searches (chunk-parallel, periodic tables)
    big = configs.make("chain_gpt_n1152_k64", batch=64)
    # second, smaller: 24 blocks of 16 strategies, one search, a non-periodic edge map
    rs = np.random.default_rng(90)
    small_cost = rs.integers(10_000, 1_000_000, size=(1, 24, 16)).astype(np.int32)
    small_rtab = rs.integers(10_000, 1_000_000, size=(5, 16, 16)).astype(np.int32)
    small_redge = rs.integers(0, 5, size=24).astype(np.int32)
    cases = [("1152x64 b64", big["cost"], big["rtab"], big["redge"]),
             ("24x16 b1", small_cost, small_rtab, small_redge)]
    for label, cost, rtab, redge in cases:
        say("noalloc", label)
        want = _reference(cost, rtab, redge)
        got = _noalloc(cost, rtab, redge)
        for name, a, b in zip(("opt", "status", "plan"), got, want):
            np.testing.assert_array_equal(a, b, err_msg=f"{name} {label}")
        assert (got[1] == 0).all()


def test_noalloc_rejects_searches_beyond_the_scratch():
    need_gpu()
    from paper_2504_00598_amd import _lib as L

    say("noalloc too large")
    rs = np.random.default_rng(91)
    B, N, K = 256, 1152, 64   # about 21 MB of argmin bytes alone, with 2048 searches beyond 32 MiB
    cost = rs.integers(0, 100, size=(8 * B, N, 16)).astype(np.int32)
    rtab = rs.integers(0, 100, size=(12, 16, 16)).astype(np.int32)
    redge = (np.arange(N) % 12).astype(np.int32)
    d = L.Desc(dev(cost), dev(rtab), redge)
    assert L.cfp_workspace_bytes(d, L.CFP_V_CHAIN) > L.CFP_NOALLOC_MAX_BYTES
    with pytest.raises(L.CfpError) as err:
        L.cfp_search_chain_noalloc(d)
    assert err.value.code == L.CFP_ERR_WORKSPACE
