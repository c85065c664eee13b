"""GPU parity of cfp_search_chain, the whole chain search (Sec. 4.4: the Eq. T
recurrence and the lowest-index optimal plan) in one call.  Small searches run
as one kernel launch that also checks the range of R and takes the edge map in
its arguments; larger ones run cfp_dp_chain and cfp_traceback.  Every case is
compared with the oracle bit for bit: optimum, status and every plan entry."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

from oracle import oracle as O
from tests.gpu_util import dev, need_gpu, oracle_threads, say
from workloads import configs, gen

pytestmark = pytest.mark.gpu

INF = gen.COST_INF


def run_search(cost, rtab, redge, ws=True):
    import torch
    from paper_2504_00598_amd import _lib as L
    d = L.Desc(dev(cost), dev(rtab), redge)
    if ws or not L.chain_search_is_one_launch(d):
        ws_t = torch.empty(L.cfp_workspace_bytes(d, L.CFP_V_CHAIN), dtype=torch.uint8, device="cuda")
        opt, st, plan = L.cfp_search_chain(d, ws=ws_t)
    else:
        opt = torch.empty(d.B, dtype=torch.int64, device="cuda")
        st = torch.empty(d.B, dtype=torch.int32, device="cuda")
        plan = torch.empty((d.B, d.N), dtype=torch.int32, device="cuda")
        L._check("cfp_search_chain", L.lib().cfp_search_chain(d.ref, None, 0, L._ptr(opt), L._ptr(st), L._ptr(plan),
                                                              L._stream(None)))
    torch.cuda.synchronize()
    return opt.cpu().numpy(), st.cpu().numpy(), plan.cpu().numpy(), L.chain_search_is_one_launch(d)


def check(cost, rtab, redge, label, one_launch=None, ws=True):
    cost = np.asarray(cost, np.int32)
    g_opt, g_st, g_plan, one = run_search(cost, rtab, redge, ws=ws)
    if one_launch is not None:
        assert one == one_launch, f"path {label}"
    o_opt, o_plan, o_st = O.chain(cost, rtab, redge, nthreads=oracle_threads())
    np.testing.assert_array_equal(g_st, o_st, err_msg=f"status {label}")
    np.testing.assert_array_equal(g_opt, o_opt, err_msg=f"opt {label}")
    np.testing.assert_array_equal(g_plan, o_plan, err_msg=f"plan {label}")
    return g_opt, g_st, g_plan


def rand_case(seed, B, N, K, E, lo, hi, rlo=None, rhi=None, inf_frac=0.0):
    rs = np.random.default_rng(seed)
    cost = rs.integers(lo, hi, size=(B, N, K)).astype(np.int32)
    if inf_frac:
        cost[rs.random((B, N, K)) < inf_frac] = INF
    rtab = rs.integers(lo if rlo is None else rlo, hi if rhi is None else rhi, size=(E, K, K)).astype(np.int32)
    redge = rs.integers(0, E, size=N).astype(np.int32)
    return cost, rtab, redge


def test_single_chain_workload():
    """The 24-block K=16 chain of one search: one launch."""
    need_gpu()
    say("search: chain_gpt_n24_k16")
    d = configs.make("chain_gpt_n24_k16")
    check(d["cost"], d["rtab"], d["redge"], "chain_gpt_n24_k16", one_launch=True)
    check(d["cost"], d["rtab"], d["redge"], "chain_gpt_n24_k16 without workspace", one_launch=True, ws=False)


# (N, K, B, E): one-row chains, K = 1, ragged K in every lane block, the longest chain,
# many searches, many tables
SHAPES = [(1, 1, 1, 1), (1, 7, 3, 2), (2, 1, 2, 1), (3, 2, 1, 1), (7, 3, 5, 3), (24, 16, 1, 12), (100, 17, 4, 6),
          (512, 16, 2, 12), (65, 32, 9, 7), (40, 33, 3, 2), (120, 48, 2, 1), (20, 64, 3, 2), (300, 20, 256, 2),
          (50, 10, 3, 40)]


@pytest.mark.parametrize("N,K,B,E", SHAPES)
def test_one_launch_shapes(N, K, B, E):
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    say("search one launch", N, K, B, E)
    rhi = min(1_000_000, cfp_r_limit(0, K))
    cost, rtab, redge = rand_case([60, N, K, B, E], B, N, K, E, 10_000, 1_000_000, rlo=0, rhi=rhi)
    check(cost, rtab, redge, f"N={N} K={K} B={B} E={E}", one_launch=True)


@pytest.mark.parametrize("N,K,B,E,one", [(82, 64, 1, 2, True), (83, 64, 1, 2, False), (95, 32, 2, 10, True),
                                         (96, 32, 2, 10, False)])
def test_lds_bound(N, K, B, E, one):
    """Both sides of the LDS bound of the one-launch path."""
    need_gpu()
    say("search LDS bound", N, K, B, E, one)
    cost, rtab, redge = rand_case([67, N, K, B, E], B, N, K, E, 10_000, 1_000_000)
    check(cost, rtab, redge, f"N={N} K={K} B={B} E={E}", one_launch=one)


@pytest.mark.parametrize("N,K,B,E", [(513, 16, 1, 12), (30, 64, 2, 12), (50, 100, 2, 3), (20, 16, 257, 2)])
def test_larger_searches_take_two_calls(N, K, B, E):
    need_gpu()
    say("search two calls", N, K, B, E)
    cost, rtab, redge = rand_case([61, N, K, B, E], B, N, K, E, 10_000, 1_000_000)
    check(cost, rtab, redge, f"N={N} K={K} B={B} E={E}", one_launch=False)


def test_ties_unavailable_and_largest_resharding():
    """Tie-heavy values (lowest index everywhere), unavailable strategies, an
    infeasible search and resharding entries at the top of the exact range."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    say("search ties")
    cost, rtab, redge = rand_case([62], 6, 60, 32, 4, 0, 3, inf_frac=0.15)
    cost[2, 40, :] = INF
    check(cost, rtab, redge, "ties", one_launch=True)
    rs = np.random.default_rng(63)
    for K in (16, 32, 64):
        lim = cfp_r_limit(0, K)
        cost = rs.integers(0, 2**31 - 1, size=(3, 20, K), dtype=np.int64).astype(np.int32)
        cost[:, :, 0] = 0
        cost[:, :, 1] = INF - 1
        rtab = rs.integers(lim - 50, lim, size=(2, K, K)).astype(np.int32)
        redge = rs.integers(0, 2, size=20).astype(np.int32)
        check(cost, rtab, redge, f"largest R K={K}", one_launch=True)


def test_bad_inputs_on_the_one_launch_path():
    """A negative cost, or a resharding entry outside [0, cfp_r_limit), gives
    BADINPUT, INT64_MAX and a plan of -1 for the searches it affects (R: all)."""
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT, CFP_ST_OK, cfp_r_limit
    say("search bad inputs")
    cost, rtab, redge = rand_case([64], 4, 30, 16, 3, 0, 1000)
    cost[1, 7, 3] = -5
    opt, st, plan, one = run_search(cost, rtab, redge)
    assert one
    assert st[1] == CFP_ST_BADINPUT and opt[1] == np.iinfo(np.int64).max and (plan[1] == -1).all()
    ok = [0, 2, 3]
    o_opt, o_plan, o_st = O.chain(cost[ok], rtab, redge, nthreads=oracle_threads())
    assert (st[ok] == CFP_ST_OK).all()
    np.testing.assert_array_equal(opt[ok], o_opt)
    np.testing.assert_array_equal(plan[ok], o_plan)
    cost[1, 7, 3] = 5
    for bad in (cfp_r_limit(0, 16), -1):
        r2 = rtab.copy()
        r2[2, 4, 9] = bad  # a table no edge uses still counts
        redge2 = (np.arange(30) % 2).astype(np.int32)
        opt, st, plan, _ = run_search(cost, r2, redge2)
        assert (st == CFP_ST_BADINPUT).all() and (opt == np.iinfo(np.int64).max).all() and (plan == -1).all()


def _device_pointer(host_tensor):
    """Device address of a pinned host tensor (hipHostGetDevicePointer), or None."""
    try:
        hip = ctypes.CDLL("libamdhip64.so")
    except OSError:
        return None
    ptr = ctypes.c_void_p()
    rc = hip.hipHostGetDevicePointer(ctypes.byref(ptr), ctypes.c_void_p(host_tensor.data_ptr()), ctypes.c_uint(0))
    return ptr.value if rc == 0 and ptr.value else None


def test_outputs_in_mapped_host_memory():
    """opt, status and plan written straight into pinned host memory, twice in a
    row on the same buffers."""
    need_gpu()
    import torch
    from paper_2504_00598_amd import _lib as L
    say("search into host memory")
    opt_h = torch.zeros(3, dtype=torch.int64, pin_memory=True)
    st_h = torch.zeros(3, dtype=torch.int32, pin_memory=True)
    plan_h = torch.zeros((3, 24), dtype=torch.int32, pin_memory=True)
    ptrs = [_device_pointer(t) for t in (opt_h, st_h, plan_h)]
    if any(p is None for p in ptrs):
        pytest.skip("pinned host memory has no device address here")
    for seed in (65, 66):
        cost, rtab, redge = rand_case([seed], 3, 24, 16, 12, 10_000, 1_000_000)
        d = L.Desc(dev(cost), dev(rtab), redge)
        L._check("cfp_search_chain", L.lib().cfp_search_chain(d.ref, None, 0, ptrs[0], ptrs[1], ptrs[2],
                                                              L._stream(None)))
        torch.cuda.synchronize()
        o_opt, o_plan, o_st = O.chain(cost, rtab, redge, nthreads=oracle_threads())
        np.testing.assert_array_equal(st_h.numpy(), o_st)
        np.testing.assert_array_equal(opt_h.numpy(), o_opt)
        np.testing.assert_array_equal(plan_h.numpy(), o_plan)
