"""GPU parity of cfp_dp_chain + cfp_traceback against the CPU oracle:
optimum, status and plan must match bit for bit."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import oracle as O
from tests.gpu_util import assert_chain_parity, dev, need_gpu, oracle_threads, run_chain, say
from workloads import configs, gen

pytestmark = pytest.mark.gpu

INF = gen.COST_INF


def rand_case(seed, B, N, K, E, lo, hi, rlo=None, rhi=None, inf_frac=0.0):
    rs = np.random.default_rng(seed)
    cost = rs.integers(lo, hi, size=(B, N, K)).astype(np.int32)
    if inf_frac:
        cost[rs.random((B, N, K)) < inf_frac] = INF
    rtab = rs.integers(lo if rlo is None else rlo, hi if rhi is None else rhi, size=(E, K, K)).astype(np.int32)
    redge = rs.integers(0, E, size=N).astype(np.int32)
    return cost, rtab, redge


@pytest.mark.parametrize("cfg", ["chain_gpt_n24_k16", "chain_gpt_n1152_k64", "chain_wide_n512_k256"])
def test_configs_full(cfg):
    need_gpu()
    say("config", cfg)
    d = configs.make(cfg)
    assert_chain_parity(d["cost"], d["rtab"], d["redge"], cfg)


SHAPES = [(1, 1), (1, 5), (2, 1), (3, 2), (7, 3), (65, 16), (130, 17), (129, 31), (64, 32), (70, 33),
          (200, 64), (66, 65), (131, 100), (90, 128), (40, 129), (67, 200), (33, 256), (20, 257), (9, 300),
          (12, 512)]


@pytest.mark.parametrize("N,K", SHAPES)
def test_shapes_realistic_values(N, K):
    need_gpu()
    say("shape", N, K)
    from paper_2504_00598_amd import cfp_r_limit
    rhi = min(10_000_000, cfp_r_limit(0, K))  # resharding values within the documented exact range
    cost, rtab, redge = rand_case([1, N, K], 3, N, K, 5, 10_000, 10_000_000, rlo=10_000, rhi=rhi)
    assert_chain_parity(cost, rtab, redge, f"N={N} K={K}")


@pytest.mark.parametrize("N,K", SHAPES)
def test_shapes_heavy_ties(N, K):
    need_gpu()
    say("ties", N, K)
    cost, rtab, redge = rand_case([2, N, K], 2, N, K, 3, 0, 3)
    assert_chain_parity(cost, rtab, redge, f"ties N={N} K={K}")


@pytest.mark.parametrize("K", [16, 64, 200, 512])
def test_largest_allowed_resharding(K):
    """R entries at cfp_r_limit - 1 and costs near 2^31: still exact."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    lim = cfp_r_limit(0, K)
    rs = np.random.default_rng(K)
    N = 50
    cost = rs.integers(2**31 - 10**6, 2**31 - 1, size=(2, N, K)).astype(np.int32)
    rtab = rs.integers(lim - 1000, lim, size=(4, K, K)).astype(np.int32)
    rtab[:, np.arange(K), np.arange(K)] = rs.integers(0, 3, size=(4, K))
    redge = rs.integers(0, 4, size=N).astype(np.int32)
    assert_chain_parity(cost, rtab, redge, f"max R K={K}")


@pytest.mark.parametrize("K", [3, 64, 256])
def test_unavailable_strategies(K):
    need_gpu()
    cost, rtab, redge = rand_case([3, K], 4, 40, K, 3, 0, 100, inf_frac=0.3)
    cost[1, 7, :] = INF        # search 1: every strategy of block 7 unavailable -> infeasible
    cost[2, 0, :] = INF        # search 2: block 0 unavailable -> infeasible
    cost[3, :, 1:] = INF       # search 3: only strategy 0 is left anywhere
    cost[3, :, 0] = 5
    g_opt, g_plan = assert_chain_parity(cost, rtab, redge, f"inf K={K}")
    assert (g_plan[1] == -1).all() and (g_plan[2] == -1).all()
    assert (g_plan[3] == 0).all()


def test_badinput_statuses():
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT, cfp_r_limit
    cost, rtab, redge = rand_case(4, 3, 20, 16, 2, 0, 100)
    cost[1, 3, 4] = -5
    opt, st, plan = run_chain(cost, rtab, redge)
    assert st.tolist() == [0, CFP_ST_BADINPUT, 0]
    assert opt[1] == np.iinfo(np.int64).max and (plan[1] == -1).all()
    rtab2 = rtab.copy()
    rtab2[1, 2, 3] = cfp_r_limit(0, 16)
    opt, st, plan = run_chain(cost, rtab2, redge)
    assert (st == CFP_ST_BADINPUT).all() and (plan == -1).all()


def test_repeat_is_bit_identical():
    need_gpu()
    d = configs.make("chain_gpt_n1152_k64", batch=32)
    first = run_chain(d["cost"], d["rtab"], d["redge"])
    for _ in range(3):
        again = run_chain(d["cost"], d["rtab"], d["redge"])
        for a, b in zip(first, again):
            np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("K", [16, 64, 100, 256])
def test_periodic_layers(K):
    """Every layer of 12 blocks repeats the same costs (profiles of one
    distinct segment reused for every instance, Sec. 4.1): a search space
    full of equal-cost plans, so the lowest-index rule decides the plan."""
    need_gpu()
    rs = np.random.default_rng(30 + K)
    B, N = 4, 240
    layer = rs.integers(0, 30, size=(B, 12, K)).astype(np.int32)
    cost = np.tile(layer, (1, N // 12, 1))
    rtab = rs.integers(0, 30, size=(12, K, K)).astype(np.int32)
    rtab[:, np.arange(K), np.arange(K)] = 0
    redge = (np.arange(N) % 12).astype(np.int32)
    say("periodic layers", K)
    assert_chain_parity(cost, rtab, redge, f"periodic K={K}")


# The traceback follows the argmin table in one launch from LDS when a search's
# table fits there (about 150 KiB: N K bytes, 2 N K for K > 256) and in three
# launches from memory otherwise; shapes on both sides of that boundary, with
# ties so that many chains of the traceback merge.
@pytest.mark.parametrize("N,K,B", [(512, 256, 2), (1152, 64, 2), (129, 512, 1), (300, 129, 2),
                                   (600, 256, 2), (2600, 64, 2), (160, 512, 1), (300, 257, 1)])
def test_traceback_lds_and_memory_paths(N, K, B):
    need_gpu()
    say("traceback path", N, K, B)
    cost, rtab, redge = rand_case([7, N, K], B, N, K, 4, 0, 50)
    assert_chain_parity(cost, rtab, redge, f"traceback N={N} K={K}")


# The chunk-parallel paths check the range of R while packing it (the other
# paths in a separate pass): an entry at cfp_r_limit or below 0 marks every
# search of the call as bad input.
@pytest.mark.parametrize("N,K,B,bad", [(400, 64, 70, "limit"), (400, 64, 70, "negative"),
                                       (200, 256, 9, "limit"), (200, 256, 9, "negative"),
                                       (20, 16, 3, "limit")])
def test_resharding_range_checked_on_every_path(N, K, B, bad):
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT, cfp_r_limit
    say("R range", N, K, B, bad)
    cost, rtab, redge = rand_case([48, N, K], B, N, K, 12, 0, 1000)
    redge = (np.arange(N) % 12).astype(np.int32)
    opt, st, plan = run_chain(cost, rtab, redge)
    assert (st == 0).all()
    rtab[7, K - 1, K // 2] = cfp_r_limit(0, K) if bad == "limit" else -1
    opt, st, plan = run_chain(cost, rtab, redge)
    assert (st == CFP_ST_BADINPUT).all() and (opt == np.iinfo(np.int64).max).all() and (plan == -1).all()


# K > 64 runs on one of two kernels: the split kernel (each search over P = K_P^2 / 4096
# workgroups, K_P the padded K, tables in registers) when all B * P workgroups fit the
# device's 256 compute units and there are at most 12 tables, else the wide kernel (one
# workgroup per search streaming its tables).  Both must give the oracle's answer.

@pytest.mark.parametrize("K,B", [(100, 65), (200, 17), (300, 5), (512, 5)])
def test_wide_path_batches(K, B):
    """Batches too large for the split kernel: the wide kernel."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    say("wide path", K, B)
    rhi = min(10_000_000, cfp_r_limit(0, K))
    cost, rtab, redge = rand_case([3, K, B], B, 40, K, 12, 10_000, 10_000_000, rlo=10_000, rhi=rhi)
    assert_chain_parity(cost, rtab, redge, f"wide K={K} B={B}")


def test_wide_path_many_tables():
    """More than 12 tables: the wide kernel even for a single search."""
    need_gpu()
    cost, rtab, redge = rand_case([4], 2, 60, 150, 17, 0, 10**6)
    assert_chain_parity(cost, rtab, redge, "wide E=17")


@pytest.mark.parametrize("N,K,B", [(300, 65, 4), (500, 128, 60), (31, 256, 16), (120, 257, 4), (127, 512, 4)])
def test_split_path_long_chains(N, K, B):
    """Few chains spread over many workgroups (B * P = 256 at the largest); the
    chains with K > 128 are too short for the chunk-parallel form."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    say("split path", N, K, B)
    rhi = min(1_000_000, cfp_r_limit(0, K))
    cost, rtab, redge = rand_case([5, N, K, B], B, N, K, 12, 10_000, 1_000_000, rlo=10_000, rhi=rhi)
    assert_chain_parity(cost, rtab, redge, f"split N={N} K={K} B={B}")


def test_long_chain_workload():
    """The 4096-block K=512 workload of the scan through the chain search (64
    chunks of 64 rows)."""
    need_gpu()
    say("config scan_n4096_k512 through cfp_dp_chain")
    d = configs.make("scan_n4096_k512")
    assert_chain_parity(d["cost"], d["rtab"], d["redge"], "long chain K=512")


# 32 < K <= 64 on long chains (at least 8 blocks of 12 rows) with at most 12 tables runs
# chunk-parallel: the chains are cut into chunks that are searched concurrently from
# arbitrary start rows and then repaired until their rows meet the speculative ones; a
# chain whose rows never meet is finished sequentially.  Whatever happens inside, the
# answer must be the oracle's.

def _no_switch_tables(rs, E, K, lim):
    """Resharding so dear that no plan ever switches strategy: the rows of two runs
    started from different rows never become parallel, so no chunk's fix-up meets
    its speculative run."""
    rtab = rs.integers(lim - 1000, lim, size=(E, K, K)).astype(np.int32)
    rtab[:, np.arange(K), np.arange(K)] = 0
    return rtab


@pytest.mark.parametrize("K,B", [(64, 3), (64, 70), (40, 9)])
def test_chunked_rows_never_meet(K, B):
    """Every chunk misses its checkpoints: the final pass reruns the chains."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    rs = np.random.default_rng([40, K, B])
    N = 600
    cost = rs.integers(0, 50, size=(B, N, K)).astype(np.int32)
    rtab = _no_switch_tables(rs, 12, K, cfp_r_limit(0, K))
    redge = (np.arange(N) % 12).astype(np.int32)
    say("chunked, no convergence", K, B)
    assert_chain_parity(cost, rtab, redge, f"never meet K={K} B={B}")


@pytest.mark.parametrize("seed", range(4))
def test_chunked_some_chunks_meet(seed):
    """A zero table (any row maps to a parallel one) placed on a few edges: chunks that
    contain one meet their speculative run, the others do not, in a seeded pattern."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    rs = np.random.default_rng([41, seed])
    K, B, N = 64, 68, 900
    cost = rs.integers(0, 1000, size=(B, N, K)).astype(np.int32)
    rtab = _no_switch_tables(rs, 3, K, cfp_r_limit(0, K))
    rtab[2] = 0
    redge = rs.integers(0, 2, size=N).astype(np.int32)
    resets = rs.choice(np.arange(1, N), size=int(rs.integers(1, 6)), replace=False)
    redge[resets] = 2
    say("chunked, partial convergence", seed, sorted(resets.tolist()))
    assert_chain_parity(cost, rtab, redge, f"partial seed={seed}")


@pytest.mark.parametrize("N,K,B", [(96, 64, 256), (100, 64, 255), (1000, 33, 67), (777, 48, 130), (1152, 64, 1),
                                   (2000, 64, 8), (481, 63, 512)])
def test_chunked_shapes(N, K, B):
    """Ragged batches (searches beyond the last full group of a workgroup), ragged last
    blocks, K below 64 and chunk counts from 2 to 64."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    rhi = min(10_000_000, cfp_r_limit(0, K))
    cost, rtab, redge = rand_case([42, N, K, B], B, N, K, 12, 10_000, 10_000_000, rlo=10_000, rhi=rhi)
    if N % 2:
        redge = (np.arange(N) % 12).astype(np.int32)  # the periodic (register-set) table selection
    say("chunked shape", N, K, B)
    assert_chain_parity(cost, rtab, redge, f"chunked N={N} K={K} B={B}")


def test_chunked_ties_and_statuses():
    """Tie-heavy values, unavailable strategies and bad inputs on the chunked path."""
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT
    cost, rtab, redge = rand_case([43], 70, 400, 64, 5, 0, 3, inf_frac=0.1)
    cost[5, 250, :] = INF   # infeasible search, in a late chunk
    assert_chain_parity(cost, rtab, redge, "chunked ties")
    cost[9, 100, 3] = -7    # a negative cost is rejected by the library (the oracle has no such check)
    opt, st, plan = run_chain(cost, rtab, redge)
    assert st[9] == CFP_ST_BADINPUT and opt[9] == np.iinfo(np.int64).max and (plan[9] == -1).all()
    assert st[5] != 0 and (st[np.r_[0:5, 6:9, 10:70]] == 0).all()


# 128 < K <= 256 on long chains (at least 32 blocks) runs chunk-parallel as well, with two
# chains per workgroup sharing each streamed table word.  Same requirement: the oracle's
# answer whatever the rows do.

@pytest.mark.parametrize("N,K,B", [(32, 256, 1), (33, 129, 2), (100, 200, 3), (513, 256, 64), (1000, 255, 5),
                                   (257, 160, 64), (64, 256, 129), (81, 256, 2)])
def test_chunked_wide_shapes(N, K, B):
    """Ragged batches (an odd last search), ragged last chunks, K below 256, one-row chunks."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    rhi = min(10_000_000, cfp_r_limit(0, K))
    cost, rtab, redge = rand_case([44, N, K, B], B, N, K, 12, 10_000, 10_000_000, rlo=10_000, rhi=rhi)
    if N % 2:
        redge = (np.arange(N) % 12).astype(np.int32)
    say("chunked wide shape", N, K, B)
    assert_chain_parity(cost, rtab, redge, f"chunked wide N={N} K={K} B={B}")


@pytest.mark.parametrize("K,B", [(256, 3), (200, 8)])
def test_chunked_wide_rows_never_meet(K, B):
    """Every chunk misses its checkpoints: the final pass reruns the chains."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    rs = np.random.default_rng([45, K, B])
    N = 300
    cost = rs.integers(0, 50, size=(B, N, K)).astype(np.int32)
    rtab = _no_switch_tables(rs, 12, K, cfp_r_limit(0, K))
    redge = (np.arange(N) % 12).astype(np.int32)
    say("chunked wide, no convergence", K, B)
    assert_chain_parity(cost, rtab, redge, f"wide never meet K={K} B={B}")


@pytest.mark.parametrize("seed", range(3))
def test_chunked_wide_some_chunks_meet(seed):
    """Zero tables on a few edges make some chunks meet and others not, in a seeded pattern."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    rs = np.random.default_rng([46, seed])
    K, B, N = 256, 6, 600
    cost = rs.integers(0, 1000, size=(B, N, K)).astype(np.int32)
    rtab = _no_switch_tables(rs, 3, K, cfp_r_limit(0, K))
    rtab[2] = 0
    redge = rs.integers(0, 2, size=N).astype(np.int32)
    resets = rs.choice(np.arange(1, N), size=int(rs.integers(1, 6)), replace=False)
    redge[resets] = 2
    say("chunked wide, partial convergence", seed, sorted(resets.tolist()))
    assert_chain_parity(cost, rtab, redge, f"wide partial seed={seed}")


def test_chunked_wide_ties_and_statuses():
    """Tie-heavy values, unavailable strategies, an infeasible search and a negative cost."""
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT
    cost, rtab, redge = rand_case([47], 9, 200, 256, 5, 0, 3, inf_frac=0.1)
    cost[4, 150, :] = INF   # infeasible search, in a late chunk
    assert_chain_parity(cost, rtab, redge, "chunked wide ties")
    cost[7, 60, 3] = -7     # a negative cost is rejected by the library
    opt, st, plan = run_chain(cost, rtab, redge)
    assert st[7] == CFP_ST_BADINPUT and opt[7] == np.iinfo(np.int64).max and (plan[7] == -1).all()
    assert st[4] != 0 and st[6] == 0 and st[8] == 0 and (st[np.r_[0:4, 5:7]] == 0).all()


def test_header_uploads_back_to_back():
    """Forty calls enqueued without a synchronisation, each with its own edge
    map and workspace: more calls than the library's ring of pinned upload
    slots, so slots are reused while earlier copies may still be queued."""
    need_gpu()
    import torch
    from paper_2504_00598_amd import search
    say("header uploads back to back")
    rs = np.random.default_rng(61)
    B, N, K, E = 2, 40, 16, 4
    rtab = rs.integers(0, 50, size=(E, K, K)).astype(np.int32)
    cases, results = [], []
    for c in range(40):
        cost = rs.integers(0, 50, size=(B, N, K)).astype(np.int32)
        redge = rs.integers(0, E, size=N).astype(np.int32)
        cases.append((cost, redge))
        results.append(search.dp_chain(dev(cost), dev(rtab), redge))
    torch.cuda.synchronize()
    for c, ((cost, redge), r) in enumerate(zip(cases, results)):
        o_opt, o_plan, o_st = O.chain(cost, rtab, redge)
        np.testing.assert_array_equal(r.opt.cpu().numpy(), o_opt, err_msg=f"opt call {c}")
        np.testing.assert_array_equal(r.plan.cpu().numpy(), o_plan, err_msg=f"plan call {c}")


def test_range_flag_does_not_leak_between_calls():
    """The chunk-parallel K=64 path with a periodic edge map does not upload the
    workspace header and flags an out-of-range R by call number: a workspace
    reused after a call with bad R, or after a call on another path, gives
    clean statuses."""
    need_gpu()
    import torch
    from paper_2504_00598_amd import CFP_ST_BADINPUT, cfp_r_limit, search
    say("range flag across calls")
    rs = np.random.default_rng(62)
    B, N, K = 70, 400, 64
    cost = rs.integers(0, 1000, size=(B, N, K)).astype(np.int32)
    rtab = rs.integers(0, 1000, size=(12, K, K)).astype(np.int32)
    periodic = (np.arange(N) % 12).astype(np.int32)
    bad = rtab.copy()
    bad[3, 5, 7] = cfp_r_limit(0, K)
    r = search.dp_chain(dev(cost), dev(bad), periodic)
    torch.cuda.synchronize()
    assert (r.status.cpu().numpy() == CFP_ST_BADINPUT).all()
    ws = r.ws
    o_opt, o_plan, o_st = O.chain(cost, rtab, periodic, nthreads=oracle_threads())
    r2 = search.dp_chain(dev(cost), dev(rtab), periodic, ws=ws)  # same workspace, good R
    torch.cuda.synchronize()
    np.testing.assert_array_equal(r2.status.cpu().numpy(), o_st)
    np.testing.assert_array_equal(r2.opt.cpu().numpy(), o_opt)
    np.testing.assert_array_equal(r2.plan.cpu().numpy(), o_plan)
    # a non-periodic edge map (another path, header uploaded) with bad R, then periodic again
    other = rs.integers(0, 12, size=N).astype(np.int32)
    r3 = search.dp_chain(dev(cost), dev(bad), other, ws=ws)
    torch.cuda.synchronize()
    assert (r3.status.cpu().numpy() == CFP_ST_BADINPUT).all()
    r4 = search.dp_chain(dev(cost), dev(rtab), periodic, ws=ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(r4.opt.cpu().numpy(), o_opt)
    np.testing.assert_array_equal(r4.plan.cpu().numpy(), o_plan)


def test_range_flag_ignores_stale_workspace_bytes():
    """The headerless K=64 path keeps its range flag in a workspace word that no
    upload clears.  Fresh workspaces whose flag word holds small integers,
    all-ones, or other leftovers (a freed plan row, an earlier cost) must still
    give a clean search."""
    need_gpu()
    import torch
    from paper_2504_00598_amd import _lib as L, search
    say("range flag with stale workspace bytes")
    rs = np.random.default_rng(63)
    B, N, K = 70, 400, 64
    cost = rs.integers(0, 1000, size=(B, N, K)).astype(np.int32)
    rtab = rs.integers(0, 1000, size=(12, K, K)).astype(np.int32)
    periodic = (np.arange(N) % 12).astype(np.int32)
    o_opt, o_plan, o_st = O.chain(cost, rtab, periodic, nthreads=oracle_threads())
    d = L.Desc(dev(cost), dev(rtab), periodic)
    nbytes = L.cfp_workspace_bytes(d, L.CFP_V_CHAIN)
    words = list(range(0, 65)) + [-1, 2**31 - 1, 2**32, 2**63 - 1, -(2**63), int(rs.integers(0, 2**62))]
    for v in words:
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        ws[:64].view(torch.int64)[:] = v   # every 8-byte word of the first 64 bytes, the flag word among them
        r = search.dp_chain(d.cost, d.rtab, periodic, ws=ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(r.status.cpu().numpy(), o_st, err_msg=f"status, stale word {v}")
        np.testing.assert_array_equal(r.opt.cpu().numpy(), o_opt, err_msg=f"opt, stale word {v}")
        np.testing.assert_array_equal(r.plan.cpu().numpy(), o_plan, err_msg=f"plan, stale word {v}")


# 256 < K <= 512 on chains of at least 128 blocks runs chunk-parallel with chunks of at
# least 64 rows (runs take tens of rows to become parallel at this width).  The final
# pass reruns, whole, each chunk that follows one whose fix-up met no checkpoint.
# Batches of at most 8 searches run in state-split teams (four workgroups per chunk,
# rows exchanged every step); larger batches carry four searches per workgroup.

@pytest.mark.parametrize("N,K,B", [(128, 512, 1), (300, 400, 5), (1000, 512, 3), (640, 300, 8), (129, 257, 2),
                                   (4096, 512, 1), (700, 512, 12), (300, 300, 9), (1200, 511, 7)])
def test_chunked_k512_shapes(N, K, B):
    """Two chunks of 64 rows, ragged K and batches, ragged last chunks, 64 chunks;
    teams of one and two groups of searches, and four searches per workgroup."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    rhi = min(1_000_000, cfp_r_limit(0, K))
    cost, rtab, redge = rand_case([48, N, K, B], B, N, K, 12, 10_000, 1_000_000, rlo=10_000, rhi=rhi)
    if N % 2 == 0:
        redge = (np.arange(N) % 12).astype(np.int32)
    say("chunked K>256 shape", N, K, B)
    assert_chain_parity(cost, rtab, redge, f"chunked K>256 N={N} K={K} B={B}")


@pytest.mark.parametrize("N,K,B", [(1089, 512, 1), (1090, 400, 5), (1091, 512, 3)])
def test_chunked_k512_short_last_chunk(N, K, B):
    """17 chunks of 68 rows and a last chunk of 1, 2 or 3 rows (a run of one
    row is its own checkpoint), in state-split teams of one and two groups."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    rhi = min(1_000_000, cfp_r_limit(0, K))
    cost, rtab, redge = rand_case([52, N, K, B], B, N, K, 12, 10_000, 1_000_000, rlo=10_000, rhi=rhi)
    say("chunked K>256, short last chunk", N, K, B)
    assert_chain_parity(cost, rtab, redge, f"short last chunk N={N} K={K} B={B}")


@pytest.mark.parametrize("K,B", [(512, 2), (300, 5)])
def test_chunked_k512_rows_never_meet(K, B):
    """No chunk meets its checkpoints: every chunk after the first is rerun in turn."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    rs = np.random.default_rng([49, K, B])
    N = 400
    cost = rs.integers(0, 50, size=(B, N, K)).astype(np.int32)
    rtab = _no_switch_tables(rs, 12, K, cfp_r_limit(0, K))
    redge = (np.arange(N) % 12).astype(np.int32)
    say("chunked K>256, no convergence", K, B)
    assert_chain_parity(cost, rtab, redge, f"K>256 never meet K={K} B={B}")


@pytest.mark.parametrize("seed", range(4))
def test_chunked_k512_some_chunks_meet(seed):
    """Zero tables on a few edges: a seeded mix of chunks that meet in the fix-up
    pass, chunks that meet only when rerun, and chunks that never meet."""
    need_gpu()
    from paper_2504_00598_amd import cfp_r_limit
    rs = np.random.default_rng([50, seed])
    K, B, N = 512, 3, 900
    cost = rs.integers(0, 1000, size=(B, N, K)).astype(np.int32)
    rtab = _no_switch_tables(rs, 3, K, cfp_r_limit(0, K))
    rtab[2] = 0
    redge = rs.integers(0, 2, size=N).astype(np.int32)
    resets = rs.choice(np.arange(1, N), size=int(rs.integers(1, 8)), replace=False)
    redge[resets] = 2
    say("chunked K>256, partial convergence", seed, sorted(resets.tolist()))
    assert_chain_parity(cost, rtab, redge, f"K>256 partial seed={seed}")


def test_teams_ignore_stale_exchange_words():
    """Batches of at most 8 searches with 256 < K <= 512 run in state-split
    teams that exchange rows as step-tagged words in the workspace.  A
    workspace of zeros (words whose tags name row 0), of all-ones, or left by
    a call on other inputs must still give the oracle's answers."""
    need_gpu()
    import torch
    from paper_2504_00598_amd import _lib as L, search
    say("teams with stale exchange words")
    rs = np.random.default_rng(64)
    B, N, K = 3, 500, 400
    runs = []
    for _ in range(2):
        cost = rs.integers(10_000, 1_000_000, size=(B, N, K)).astype(np.int32)
        rtab = rs.integers(10_000, 1_000_000, size=(12, K, K)).astype(np.int32)
        rtab[:, np.arange(K), np.arange(K)] = 0
        redge = rs.integers(0, 12, size=N).astype(np.int32)
        o_opt, o_plan, o_st = O.chain(cost, rtab, redge, nthreads=oracle_threads())
        runs.append((dev(cost), dev(rtab), redge, o_opt, o_plan, o_st))
    nbytes = L.cfp_workspace_bytes(L.Desc(runs[0][0], runs[0][1], runs[0][2]), L.CFP_V_CHAIN)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    for fill in (0, 0xFF, 0x01):
        ws.fill_(fill)
        for j in (0, 1, 0):
            c, r, e, o_opt, o_plan, o_st = runs[j]
            res = search.dp_chain(c, r, e, ws=ws)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(res.status.cpu().numpy(), o_st, err_msg=f"status, fill {fill} input {j}")
            np.testing.assert_array_equal(res.opt.cpu().numpy(), o_opt, err_msg=f"opt, fill {fill} input {j}")
            np.testing.assert_array_equal(res.plan.cpu().numpy(), o_plan, err_msg=f"plan, fill {fill} input {j}")


def test_chunked_k512_ties_and_statuses():
    """Tie-heavy values, unavailable strategies, an infeasible search and a negative cost."""
    need_gpu()
    from paper_2504_00598_amd import CFP_ST_BADINPUT
    cost, rtab, redge = rand_case([51], 5, 300, 512, 5, 0, 3, inf_frac=0.1)
    cost[2, 250, :] = INF   # infeasible search, in a late chunk
    assert_chain_parity(cost, rtab, redge, "chunked K>256 ties")
    cost[4, 70, 3] = -7     # a negative cost is rejected by the library
    opt, st, plan = run_chain(cost, rtab, redge)
    assert st[4] == CFP_ST_BADINPUT and opt[4] == np.iinfo(np.int64).max and (plan[4] == -1).all()
    assert st[2] != 0 and (st[[0, 1, 3]] == 0).all()
