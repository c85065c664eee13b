"""GPU parity of cfp_dp_segments + cfp_traceback_segments (segment-level
search with boundary-pair resharding) against the oracle: the chain search
over the expanded K x K tables.  Optimum, status and plan bit for bit."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import oracle as O
from tests.gpu_util import dev, need_gpu, oracle_threads, say
from workloads import configs, gen

pytestmark = pytest.mark.gpu
INF = gen.COST_INF


def run_seg(cost, rbound, last, first, redge):
    import torch
    from paper_2504_00598_amd import search
    res = search.dp_segments(dev(cost), dev(rbound), dev(np.asarray(last, np.uint8)),
                             dev(np.asarray(first, np.uint8)), redge)
    torch.cuda.synchronize()
    return res.opt.cpu().numpy(), res.status.cpu().numpy(), res.plan.cpu().numpy()


def assert_seg_parity(cost, rbound, last, first, redge, label=""):
    cost = np.asarray(cost, np.int32)
    if cost.ndim == 2:
        cost = cost[None]
    g_opt, g_st, g_plan = run_seg(cost, rbound, last, first, redge)
    o_opt, o_plan, o_st = O.segments(cost, rbound, last, first, redge, nthreads=oracle_threads())
    np.testing.assert_array_equal(g_st, o_st, err_msg=f"status {label}")
    np.testing.assert_array_equal(g_opt, o_opt, err_msg=f"opt {label}")
    np.testing.assert_array_equal(g_plan, o_plan, err_msg=f"plan {label}")
    return g_opt, g_plan


def seg_case(seed, B, N, P, S, E, lo, hi):
    rs = np.random.default_rng(seed)
    K = S ** P
    last, first = gen.digit_maps(P, S)
    cost = rs.integers(lo, hi, size=(B, N, K)).astype(np.int32)
    # boundary entries inside the exact range for this K (2^23 - 1 at K = 512)
    rhi = min(hi, (1 << (32 - max(4, int(np.ceil(np.log2(K)))))) - 1)
    rbound = rs.integers(min(lo, rhi - 1), rhi, size=(E, S, S)).astype(np.int32)
    redge = rs.integers(0, E, size=N).astype(np.int32)
    return cost, rbound, last, first, redge


def test_config_full():
    need_gpu()
    say("config seg_gpt_n96_k81")
    d = configs.make("seg_gpt_n96_k81")
    assert_seg_parity(d["cost"], d["rbound"], d["last"], d["first"], d["redge"], "seg config")


# K = S^P spans every kernel shape: states per lane 1, 2, 4, 8 (K up to 64, 128, 256, 512) with up to
# 4 or up to 8 boundary strategies; N = 9 and 17 end one row into a group of 8 steps
@pytest.mark.parametrize("N,P,S", [(1, 1, 2), (2, 1, 5), (5, 2, 3), (50, 4, 3), (30, 3, 4), (20, 5, 2), (40, 4, 4),
                                   (10, 2, 8), (8, 3, 8), (70, 2, 7), (25, 3, 6), (12, 9, 2), (9, 4, 3),
                                   (17, 2, 3)])
def test_shapes(N, P, S):
    need_gpu()
    say("seg shape", N, P, S)
    cost, rbound, last, first, redge = seg_case([N, P, S], 5, N, P, S, 3, 10_000, 10_000_000)
    assert_seg_parity(cost, rbound, last, first, redge, f"N={N} P={P} S={S}")


def test_general_maps_unequal_boundaries():
    """Arbitrary plan-to-boundary maps with different strategy counts on the
    two sides (L = 3 last-block strategies, F = 5 first-block ones)."""
    need_gpu()
    rs = np.random.default_rng(77)
    B, N, K, L, F = 6, 60, 100, 3, 5
    last = rs.integers(0, L, size=K).astype(np.uint8)
    first = rs.integers(0, F, size=K).astype(np.uint8)
    cost = rs.integers(0, 10**6, size=(B, N, K)).astype(np.int32)
    rbound = rs.integers(0, 10**6, size=(4, L, F)).astype(np.int32)
    redge = rs.integers(0, 4, size=N).astype(np.int32)
    assert_seg_parity(cost, rbound, last, first, redge, "general maps")


@pytest.mark.parametrize("S", [2, 3])
def test_heavy_ties(S):
    need_gpu()
    cost, rbound, last, first, redge = seg_case([9, S], 8, 40, 4, S, 2, 0, 3)
    assert_seg_parity(cost, rbound, last, first, redge, f"ties S={S}")


def test_unavailable_and_statuses():
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT, CFP_ST_INFEASIBLE, cfp_r_limit, CFP_V_SEG
    cost, rbound, last, first, redge = seg_case(10, 4, 20, 4, 3, 2, 0, 1000)
    cost[0][cost[0] % 4 == 0] = INF
    cost[1, 7, :] = INF                     # no plan
    cost[2, 3, 5] = -1                      # negative cost
    opt, st, plan = run_seg(cost, rbound, last, first, redge)
    assert st[1] == CFP_ST_INFEASIBLE and st[2] == CFP_ST_BADINPUT
    assert (plan[1] == -1).all() and (plan[2] == -1).all()
    assert_seg_parity(cost[[0, 3]], rbound, last, first, redge, "inf")
    # boundary entry at the exact-range limit, and a map entry out of range
    rb = rbound.copy()
    rb[1, 2, 0] = cfp_r_limit(CFP_V_SEG, 81)
    _, st, _ = run_seg(cost[[0, 3]], rb, last, first, redge)
    assert (st == CFP_ST_BADINPUT).all()
    bad_last = last.copy()
    bad_last[17] = 3
    _, st, _ = run_seg(cost[[0, 3]], rbound, bad_last, first, redge)
    assert (st == CFP_ST_BADINPUT).all()
    bad_first = first.copy()
    bad_first[80] = 3
    _, st, _ = run_seg(cost[[0, 3]], rbound, last, bad_first, redge)
    assert (st == CFP_ST_BADINPUT).all()


def test_max_boundary_values():
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit, CFP_V_SEG
    cost, rbound, last, first, redge = seg_case(11, 4, 64, 4, 3, 2, 0, 10**7)
    rbound[:] = cfp_r_limit(CFP_V_SEG, 81) - 1
    rbound[:, np.arange(3), np.arange(3)] = 0
    assert_seg_parity(cost, rbound, last, first, redge, "max r")


def test_repeat_is_bit_identical():
    need_gpu()
    d = configs.make("seg_gpt_n96_k81", batch=32)
    a = run_seg(d["cost"], d["rbound"], d["last"], d["first"], d["redge"])
    for _ in range(3):
        b = run_seg(d["cost"], d["rbound"], d["last"], d["first"], d["redge"])
        for x, y in zip(a, b):
            np.testing.assert_array_equal(x, y)


# Batches that leave SIMDs idle run each chain as chunks (rank convergence): one
# workgroup per search, P = min(8, 1024 // B, N // 16) chunks of ceil(N / P) rows.
def seg_chunks(N, B):
    P = min(8, max(1, 1024 // B), N // 16)
    return P if P >= 2 else 1


def test_chunked_shapes_across_kernel_forms():
    """The chunked path at K = 512 (16-bit argmins, eight states per lane) and
    at K = 216 with six boundary strategies (the eight-class form)."""
    need_gpu()
    for seed, (B, N, P, S) in enumerate([(3, 40, 9, 2), (4, 48, 3, 6), (2, 64, 4, 3)]):
        say("seg chunked", B, N, P, S)
        assert seg_chunks(N, B) >= 2
        cost, rbound, last, first, redge = seg_case([70, seed], B, N, P, S, 3, 10_000, 10_000_000)
        assert_seg_parity(cost, rbound, last, first, redge, f"chunked B={B} N={N} K={S ** P}")


def _class_chains(seed, B, N, E_mix, pattern):
    """Plans whose first and last block strategies coincide (first = last = s mod 3) and
    boundary table 0 that never moves a search between classes (0 on the diagonal, the
    largest entry off it): over rows using table 0 the three classes run as separate
    chains, so a run started anywhere else never becomes parallel to the true one.  The
    other tables mix the classes.  pattern[p] says whether chunk p's rows use table 0."""
    from paper_2504_00598_amd import cfp_r_limit, CFP_V_SEG
    rs = np.random.default_rng(seed)
    K, L = 12, 3
    last = (np.arange(K) % L).astype(np.uint8)
    first = last.copy()
    cost = rs.integers(0, 10**6, size=(B, N, K)).astype(np.int32)
    rbound = rs.integers(0, 10**5, size=(1 + E_mix, L, L)).astype(np.int32)
    rbound[0] = cfp_r_limit(CFP_V_SEG, K) - 1
    rbound[0][np.arange(L), np.arange(L)] = 0
    P = seg_chunks(N, B)
    CL = -(-N // P)
    redge = rs.integers(1, 1 + E_mix, size=N).astype(np.int32)
    for p, iso in enumerate(pattern):
        if iso:
            redge[p * CL:min((p + 1) * CL, N)] = 0
    return cost, rbound, last, first, redge, P


def test_chunked_rows_that_never_meet():
    """Every row's table keeps the classes apart: no fix-up meets its chunk's
    speculative rows, and the final pass reruns every chunk after the first."""
    need_gpu()
    say("seg chunks never meet")
    cost, rbound, last, first, redge, P = _class_chains(71, 4, 64, 2, [True] * 8)
    assert P == 4
    assert_seg_parity(cost, rbound, last, first, redge, "never meet")


@pytest.mark.parametrize("pattern", [(False, True, False, False), (False, True, True, False),
                                     (True, False, True, False), (False, False, False, True)])
def test_chunked_rows_that_meet_in_some_chunks(pattern):
    """A chunk of class-separating rows leaves its successor's fix-up started from a
    wrong row: that chunk is rerun from the true row, at least as far as its fix-up
    went, and where the rerun meets the speculative rows the chunks after it count
    again; two such chunks in a row chain the reruns."""
    need_gpu()
    say("seg chunks meet in some", pattern)
    cost, rbound, last, first, redge, P = _class_chains([72, *pattern], 4, 64, 2, pattern)
    assert P == 4
    assert_seg_parity(cost, rbound, last, first, redge, f"pattern {pattern}")


@pytest.mark.parametrize("B,N,P,S", [(3, 1600, 2, 3), (520, 1600, 2, 2), (520, 50, 2, 3)])
def test_edge_map_in_arguments_and_in_workspace(B, N, P, S):
    """Chains of up to 1536 segments carry their edge map in the kernel
    arguments; longer ones read the device copy uploaded with the header.  Both,
    chunked (small batch) and one wave per search (B >= 512)."""
    need_gpu()
    say("seg edge map", B, N, P, S)
    cost, rbound, last, first, redge = seg_case([73, B, N], B, N, P, S, 5, 10_000, 10_000_000)
    assert_seg_parity(cost, rbound, last, first, redge, f"B={B} N={N} K={S ** P}")
