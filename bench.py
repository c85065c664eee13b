"""Benchmark of the chain search on one MI355X.

A step is one whole search of the batched chain workload (N=1152 blocks,
K=64 strategies, 256 independent searches, 12 shared resharding tables): the
forward min-plus pass plus the traceback of every plan, with all inputs
already resident in device memory.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--no-cpu]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "min-plus cell updates/sec (K² per block per search) + search latency"
# VALU roofline: 256 CUs x 64 lanes x 2.4 GHz = 39.32e12 32-bit lane-ops/s; a
# min-plus cell needs one add and one min, and gfx950 does two cells in
# three instructions (two saturating adds + one three-input min).
VALU_LANE_OPS = 256 * 64 * 2.4e9
INSTR_PER_CELL = 1.5
PEAK_CELLS = VALU_LANE_OPS / INSTR_PER_CELL
DEFAULT_CONFIG = "chain_gpt_n1152_k64"


def cells_of(cfg) -> int:
    """Min-plus cell updates of one pass: (N-1) steps of K*K per search."""
    return cfg.B * (cfg.N - 1) * cfg.K * cfg.K


def cpu_baseline(cfg, data, budget_s: float = 20.0) -> dict:
    """The oracle (plain C, one search per thread) on a bounded sample."""
    from oracle import oracle as O

    threads = max(1, min(os.cpu_count() or 1, cfg.B))
    per_search = (cfg.N - 1) * cfg.K * cfg.K
    # size the sample to about budget_s seconds at ~1 ns per cell per thread
    n = int(min(cfg.B, max(threads, budget_s * 1e9 * threads / per_search / 4)))
    t0 = time.perf_counter()
    O.chain(data["cost"][:n], data["rtab"], data["redge"], nthreads=min(threads, n))
    dt = time.perf_counter() - t0
    return {"value": n * per_search / dt, "unit": "cell/s", "cores": min(threads, n), "kind": "oracle",
            "sample": f"{n} of {cfg.B} searches of {cfg.name} (forward + traceback), {dt:.2f} s"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default=DEFAULT_CONFIG)
    ap.add_argument("--no-cpu", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the search batch is not sharded across GPUs "
              "(searches are independent; a multi-GPU run would split the batch).", file=sys.stderr)
        return 2

    import torch

    from paper_2504_00598_amd import _lib as L
    from workloads import configs

    cfg = configs.BY_NAME[args.config]
    if cfg.form != "chain":
        print("bench.py times the chain workloads; use the parity tests for the others", file=sys.stderr)
        return 2
    data = configs.make(cfg)
    cost = torch.from_numpy(data["cost"]).cuda()
    rtab = torch.from_numpy(data["rtab"]).cuda()
    desc = L.Desc(cost, rtab, data["redge"])
    ws = torch.empty(L.cfp_workspace_bytes(desc, L.CFP_V_CHAIN), dtype=torch.uint8, device="cuda")
    opt = torch.empty(cfg.B, dtype=torch.int64, device="cuda")
    status = torch.empty(cfg.B, dtype=torch.int32, device="cuda")
    plan = torch.empty((cfg.B, cfg.N), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        L.cfp_dp_chain(desc, ws=ws, opt=opt, status=status, stream=stream)
        L.cfp_traceback(desc, L.CFP_V_CHAIN, ws, plan=plan, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, m, b in ev:
        a.record(stream)
        L.cfp_dp_chain(desc, ws=ws, opt=opt, status=status, stream=stream)
        m.record(stream)
        L.cfp_traceback(desc, L.CFP_V_CHAIN, ws, plan=plan, stream=stream)
        b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fwd_ms = float(np.mean([a.elapsed_time(m) for a, m, _ in ev]))
    tb_ms = float(np.mean([m.elapsed_time(b) for _, m, b in ev]))
    ms_per_step = wall * 1e3 / args.steps

    cells = cells_of(cfg)
    value = cells / (ms_per_step * 1e-3)
    fwd_cells_s = cells / (fwd_ms * 1e-3)

    # search latency of the single-chain workload (N=24, K=16, batch 1): forward + traceback + sync
    small = configs.make("chain_gpt_n24_k16")
    sc = torch.from_numpy(small["cost"]).cuda()
    sr = torch.from_numpy(small["rtab"]).cuda()
    sd = L.Desc(sc, sr, small["redge"])
    sws = torch.empty(L.cfp_workspace_bytes(sd, L.CFP_V_CHAIN), dtype=torch.uint8, device="cuda")
    lat = []
    for it in range(60):
        t = time.perf_counter()
        o, s_, _ = L.cfp_dp_chain(sd, ws=sws, stream=stream)
        p = L.cfp_traceback(sd, L.CFP_V_CHAIN, sws, stream=stream)
        p.cpu()
        if it >= 10:
            lat.append((time.perf_counter() - t) * 1e6)

    # parity of this run's answer with the oracle (whole batch)
    from oracle import oracle as O

    o_opt, o_plan, o_st = O.chain(data["cost"], data["rtab"], data["redge"],
                                  nthreads=max(1, min(16, os.cpu_count() or 1)))
    parity = bool(np.array_equal(opt.cpu().numpy(), o_opt) and np.array_equal(plan.cpu().numpy(), o_plan)
                  and np.array_equal(status.cpu().numpy(), o_st))

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "cell/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "blocks": cfg.N, "strategies": cfg.K, "searches": cfg.B,
                   "resharding_tables": 12},
        "forward_ms": fwd_ms,
        "traceback_ms": tb_ms,
        "search_latency_us": {"workload": "chain_gpt_n24_k16", "median": float(np.median(lat)),
                              "p10": float(np.percentile(lat, 10)), "p90": float(np.percentile(lat, 90))},
        "parity_vs_oracle": parity,
        "roofline": {"bound": "alu", "achieved": fwd_cells_s / 1e12, "peak": PEAK_CELLS / 1e12,
                     "unit": "Tcell/s", "frac": fwd_cells_s / PEAK_CELLS, "traffic": None},
    }
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(cfg, data)
    print(json.dumps(out), flush=True)
    return 0 if parity else 1


if __name__ == "__main__":
    sys.exit(main())
