"""Benchmark of the plan search on one MI355X.

A step is one whole search of a batch of synthetic chains: the forward pass
plus the traceback of every plan, with every input already resident in
device memory.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--no-cpu]

By default every workload is timed in turn and the line carries one record
per workload under "configs"; the headline figures are those of the largest,
scan_n4096_k512 (4096 blocks, 512 strategies, 4 searches, the min-plus
parallel-scan form).  The records also hold the budget frontier of the memory
workload and the scan workload run through the chain search.
With --config only that workload is timed: chain_gpt_n24_k16,
chain_gpt_n1152_k64, mem_llama_n288_k32 (with --frontier: every budget in one
pass), chain_wide_n512_k256, scan_n4096_k512 (with --chain: the chain
search), seg_gpt_n96_k81 (segment-level search with boundary resharding).
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
# three instructions (two adds + one three-input min).
VALU_LANE_OPS = 256 * 64 * 2.4e9
INSTR_PER_CELL = 1.5
PEAK_CELLS = VALU_LANE_OPS / INSTR_PER_CELL


# The kernel that dominates the forward pass of each workload, and the source
# files it is built from.
# What the dominant kernel's figure covers, where it is not the whole forward call.
KERNEL_ROLE = {
    "chain_gpt_n24_k16": "the whole search (forward pass and traceback) in one launch",
    "chain_gpt_n1152_k64": "speculative pass only; forward_call_frac covers the whole forward call",
    "chain_wide_n512_k256": "speculative pass only; forward_call_frac covers the whole forward call",
    "scan_n4096_k512:chain": "speculative pass only (four workgroups per chunk, rows exchanged every step); "
                             "forward_call_frac covers the whole forward call",
    "scan_n4096_k512": "the 12 min-plus matrix-product launches of the up-sweep",
    "seg_gpt_n96_k81": "the forward pass in one launch (speculative, fix-up and final passes of four chunks per search)",
}
KERNELS = {
    # one launch of cfp_search_chain: forward pass and traceback
    "chain_gpt_n24_k16": ("chain_small_kernel<16>", ["chain_small.hip"]),
    # speculative pass of the chunk-parallel search: it computes every step of every chain
    "chain_gpt_n1152_k64": ("chain_wave_kernel<12>", ["chain_wave.hip", "res_common.h"]),
    "mem_llama_n288_k32": ("mem_fwd_kernel<32>", ["mem_fwd.hip", "res_common.h"]),
    # speculative pass of the chunk-parallel search
    "chain_wide_n512_k256": ("chain_cw_kernel<256,0>", ["chain_cw.hip", "chain_fwd_wide.hip"]),
    # the scan workload through the chain search: speculative pass of the chunk-parallel form
    "scan_n4096_k512:chain": ("chain_cx_kernel<0>", ["chain_cw.hip", "chain_fwd_wide.hip"]),
    "scan_n4096_k512": ("scan_gemm_kernel", ["scan.hip"]),
    "seg_gpt_n96_k81": ("seg_chunk_kernel<2, 4, true>", ["seg_fwd.hip"]),
}
COMMON_SOURCES = ["common.h", "cfp_internal.h", "../../include/cfp.h"]

# HBM bytes per launch of the dominant kernel, from two rocprofv3 --pmc runs
# of this script (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch), each scaled
# by the factor that maps the counter onto the bytes of a plain 512 MiB copy
# (bench.py --calibrate-copy: FETCH_SIZE reads 262167 KiB -> x2.000,
# WRITE_SIZE reads 524288 KiB -> x1.000).  "sources" is sources_hash() of the
# kernel when the counters were taken; a different hash means the kernel has
# changed and the figure is withheld.
FETCH_SCALE, WRITE_SCALE = 524288.0 / 262166.9, 524288.0 / 524288.0
TRAFFIC = {
    "chain_gpt_n24_k16": {"fetch_kib": 12.7, "write_kib": 0.2, "sources": "52818aaa4e4934d4"},
    "chain_gpt_n1152_k64": {"fetch_kib": 37976.1, "write_kib": 37516.8, "sources": "7611dbd3b031e2fb"},
    "mem_llama_n288_k32": {"fetch_kib": 127247.8, "write_kib": 338789.8, "sources": "800a6f06f2b6bf9f"},
    "chain_wide_n512_k256": {"fetch_kib": 45109.3, "write_kib": 16423.7, "sources": "fabd52fde0631d42"},
    # mean over the 12 matrix-product launches of one forward call
    "scan_n4096_k512": {"fetch_kib": 3034309.5, "write_kib": 1398442.5, "sources": "2746a9b212acf5ef"},
    "seg_gpt_n96_k81": {"fetch_kib": 6338.9, "write_kib": 10137.1, "sources": "1d03d894fb522632"},
    # the memory workload run as a budget frontier (every chunk of every search active)
    "mem_llama_n288_k32:frontier": {"fetch_kib": 166120.7, "write_kib": 442222.8, "sources": "800a6f06f2b6bf9f"},
    # the scan workload through the chain search (speculative pass)
    "scan_n4096_k512:chain": {"fetch_kib": 290919.0, "write_kib": 89986.2, "sources": "fabd52fde0631d42"},
}


def sources_hash(config: str) -> str:
    """Hash of the kernel's sources with comments and blank space removed, so
    that only a change of code withholds the traffic figure."""
    import hashlib
    import re

    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2504_00598_amd", "csrc")
    for f in KERNELS[config][1] + COMMON_SOURCES:
        with open(os.path.join(csrc, f)) as fh:
            code = re.sub(r"/\*.*?\*/", " ", fh.read(), flags=re.S)
        code = re.sub(r"//[^\n]*", " ", code)
        h.update(" ".join(code.split()).encode())
    return h.hexdigest()[:16]


def traffic_bytes(config: str, mode: str = ""):
    key = config + (":" + mode if mode else "")
    t = TRAFFIC.get(key)
    if t is None or t["sources"] != sources_hash(key if key in KERNELS else config):
        return None
    return (t["fetch_kib"] * FETCH_SCALE + t["write_kib"] * WRITE_SCALE) * 1024.0


def oracle_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def cells_of(cfg, data) -> int:
    """Min-plus cell updates of one pass, K*K per block step per search (and
    per memory bucket within the budget for the memory variant)."""
    steps = cfg.N - 1
    if cfg.form == "mem":
        return int(sum(steps * cfg.K * cfg.K * (int(bb) + 1) for bb in data["budget"]))
    return cfg.B * steps * cfg.K * cfg.K


def scan_gemm_cells(cfg) -> int:
    """Cells of the scan's min-plus matrix products: N-1 products of K^3."""
    return cfg.B * (cfg.N - 1) * cfg.K ** 3


def run_oracle(cfg, data, n=None, threads=None):
    from oracle import oracle as O

    n = cfg.B if n is None else n
    threads = threads or oracle_threads()
    if cfg.form == "mem":
        return O.chain_mem(data["cost"][:n], data["rtab"], data["redge"], data["mem"][:n], data["budget"][:n],
                           nthreads=threads)
    if cfg.form == "seg":
        return O.segments(data["cost"][:n], data["rbound"], data["last"], data["first"], data["redge"],
                          nthreads=threads)
    return O.chain(data["cost"][:n], data["rtab"], data["redge"], nthreads=threads)


def oracle_parity(cfg, data, g) -> bool:
    """The GPU results of the whole workload against the oracle's: optimum,
    status and every plan entry (and, for the frontier, every budget)."""
    o_opt, o_plan, o_st = run_oracle(cfg, data)
    ok = bool(np.array_equal(g["opt"], o_opt) and np.array_equal(g["plan"], o_plan)
              and np.array_equal(g["status"], o_st))
    if g.get("frontier") is not None:
        from oracle import oracle as O

        ok = ok and bool(np.array_equal(
            g["frontier"],
            O.mem_frontier(data["cost"], data["rtab"], data["redge"], data["mem"], cfg.M, nthreads=oracle_threads())))
    return ok


def cpu_baseline(cfg, data, budget_s: float = 10.0) -> dict:
    """The oracle (plain C, int64, one search per thread) on a bounded sample:
    whole searches of the same workload, repeated until about budget_s."""
    threads = max(1, min(os.cpu_count() or 1, cfg.B))
    per_search = cells_of(cfg, data) / cfg.B
    n = cfg.B
    t0 = time.perf_counter()
    run_oracle(cfg, data, n=min(n, threads), threads=threads)
    first = time.perf_counter() - t0
    # as many whole searches as fit the budget (at least one round of threads)
    n = int(min(cfg.B, max(threads, threads * budget_s / max(first, 1e-6) / 2)))
    reps, done, t0 = 0, 0, time.perf_counter()
    while True:
        run_oracle(cfg, data, n=n, threads=min(threads, n))
        reps += 1
        done += n
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    return {"value": done * per_search / dt, "unit": "cell/s", "cores": min(threads, n), "kind": "oracle",
            "sample": f"{reps} x {n} of {cfg.B} searches of {cfg.name} (forward + traceback), {dt:.2f} s"}


class Runner:
    """Device buffers and the two calls of one search pass.  With frontier=True
    (memory workload) the forward pass is the budget frontier: the least cost
    at every budget 0 .. M-1, and the traceback returns the plans at M-1.  A
    chain search small enough for the one-launch path of cfp_search_chain runs
    as that one call (forward pass and traceback together, the traceback step
    then empty)."""

    def __init__(self, cfg, data, frontier: bool = False):
        import torch

        from paper_2504_00598_amd import _lib as L

        self.L, self.cfg = L, cfg
        self.cost = cost = torch.from_numpy(data["cost"]).cuda()
        self.stream = torch.cuda.current_stream()
        self.opt = torch.empty(cfg.B, dtype=torch.int64, device="cuda")
        self.status = torch.empty(cfg.B, dtype=torch.int32, device="cuda")
        self.plan = torch.empty((cfg.B, cfg.N), dtype=torch.int32, device="cuda")
        self.frontier = None
        if cfg.form == "seg":
            self.variant = L.CFP_V_SEG
            self.sdesc = L.SegDesc(cost, torch.from_numpy(data["rbound"]).cuda(),
                                   torch.from_numpy(data["last"]).cuda(), torch.from_numpy(data["first"]).cuda(),
                                   data["redge"])
            self.ws = torch.empty(L.cfp_segment_workspace_bytes(self.sdesc), dtype=torch.uint8, device="cuda")
            return
        rtab = torch.from_numpy(data["rtab"]).cuda()
        self.desc = L.Desc(cost, rtab, data["redge"])
        self.variant = {"chain": L.CFP_V_CHAIN, "mem": L.CFP_V_MEM, "scan": L.CFP_V_SCAN}[cfg.form]
        self.n_mem = cfg.M if cfg.form == "mem" else 0
        if cfg.form == "mem":
            self.mem = torch.from_numpy(data["mem"]).cuda()
            self.budget = torch.from_numpy(data["budget"]).cuda()
        self.ws = torch.empty(L.cfp_workspace_bytes(self.desc, self.variant, self.n_mem), dtype=torch.uint8,
                              device="cuda")
        self.one_call = cfg.form == "chain" and L.chain_search_is_one_launch(self.desc)
        if frontier:
            if cfg.form != "mem":
                raise ValueError("the budget frontier needs the memory workload")
            self.frontier = torch.empty((cfg.B, cfg.M), dtype=torch.int64, device="cuda")

    def forward(self):
        L = self.L
        if self.variant == L.CFP_V_SEG:
            L.cfp_dp_segments(self.sdesc, ws=self.ws, opt=self.opt, status=self.status, stream=self.stream)
        elif self.variant == L.CFP_V_CHAIN and self.one_call:
            L.cfp_search_chain(self.desc, ws=self.ws, opt=self.opt, status=self.status, plan=self.plan,
                               stream=self.stream)
        elif self.variant == L.CFP_V_CHAIN:
            L.cfp_dp_chain(self.desc, ws=self.ws, opt=self.opt, status=self.status, stream=self.stream)
        elif self.frontier is not None:
            L.cfp_mem_frontier(self.desc, self.mem, self.n_mem, ws=self.ws, frontier=self.frontier,
                               status=self.status, stream=self.stream)
        elif self.variant == L.CFP_V_MEM:
            L.cfp_dp_chain_mem(self.desc, self.mem, self.n_mem, self.budget, ws=self.ws, opt=self.opt,
                               status=self.status, stream=self.stream)
        else:
            L.cfp_minplus_scan(self.desc, ws=self.ws, opt=self.opt, status=self.status, stream=self.stream)

    def traceback(self):
        if getattr(self, "one_call", False):
            return
        if self.variant == self.L.CFP_V_SEG:
            self.L.cfp_traceback_segments(self.sdesc, self.ws, plan=self.plan, stream=self.stream)
            return
        self.L.cfp_traceback(self.desc, self.variant, self.ws, n_mem=self.n_mem, plan=self.plan, stream=self.stream)


def pcie_inclusive(r, data, reps: int = 5) -> dict:
    """Whole-job rate when the cost (and mem) tables start in pinned host
    memory and the plans end there: host-to-device copy + forward + traceback
    + device-to-host copy of the plans, wall time per pass."""
    import torch

    host = {"cost": torch.from_numpy(data["cost"]).pin_memory()}
    if r.cfg.form == "mem":
        host["mem"] = torch.from_numpy(data["mem"]).pin_memory()
    plan = torch.empty(tuple(r.plan.shape), dtype=torch.int32).pin_memory()
    dt = []
    for it in range(reps + 1):
        torch.cuda.synchronize()
        t = time.perf_counter()
        r.cost.copy_(host["cost"], non_blocking=True)
        if "mem" in host:
            r.mem.copy_(host["mem"], non_blocking=True)
        r.forward()
        r.traceback()
        plan.copy_(r.plan, non_blocking=True)
        torch.cuda.synchronize()
        if it:
            dt.append(time.perf_counter() - t)
    ms = float(np.median(dt)) * 1e3
    return {"ms_per_pass": ms, "cell_per_s": cells_of(r.cfg, data) / (ms * 1e-3),
            "host_bytes": int(sum(v.numel() * v.element_size() for v in host.values()) + plan.numel() * 4)}


def _host_device_pointer(host_tensor):
    """Device address of a pinned host tensor (hipHostGetDevicePointer), or None."""
    import ctypes

    hip = ctypes.CDLL("libamdhip64.so")
    ptr = ctypes.c_void_p()
    rc = hip.hipHostGetDevicePointer(ctypes.byref(ptr), ctypes.c_void_p(host_tensor.data_ptr()), ctypes.c_uint(0))
    return ptr.value if rc == 0 and ptr.value else None


def search_latency_us(stream) -> dict:
    """Wall time of one whole search of the single-chain workload (N=24, K=16,
    one search), from the call until the plan is readable on the host: one
    cfp_search_chain call (one kernel launch: range checks, forward pass and
    traceback) writing opt, status and plan into pinned host memory mapped
    into the device.  The caller learns that the answer is there in one of two
    ways, both timed: it polls the status word, which the kernel writes last
    after a system-scope fence (`median`), or it synchronises the stream
    (`median_stream_sync`).  If the pinned memory has no device address, the
    outputs go to device memory, are copied back and the stream is
    synchronised."""
    import ctypes

    import torch

    from paper_2504_00598_amd import _lib as L
    from workloads import configs

    small = configs.make("chain_gpt_n24_k16")
    sd = L.Desc(torch.from_numpy(small["cost"]).cuda(), torch.from_numpy(small["rtab"]).cuda(), small["redge"])
    opt_h = torch.zeros(sd.B, dtype=torch.int64, pin_memory=True)
    st_h = torch.zeros(sd.B, dtype=torch.int32, pin_memory=True)
    plan_h = torch.zeros((sd.B, sd.N), dtype=torch.int32, pin_memory=True)
    ptrs = [_host_device_pointer(t) for t in (opt_h, st_h, plan_h)]
    mapped = all(p is not None for p in ptrs)
    if not mapped:
        dbufs = (torch.empty_like(opt_h, device="cuda"), torch.empty_like(st_h, device="cuda"),
                 torch.empty_like(plan_h, device="cuda"))
        ptrs = [t.data_ptr() for t in dbufs]
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipStreamSynchronize.argtypes = [ctypes.c_void_p]
    search = L.lib().cfp_search_chain
    ref, sp = sd.ref, L._stream(stream)
    st_np = st_h.numpy()

    def run(poll: bool, calls: int):
        lat = []
        for it in range(calls + 10):
            st_np[0] = -1
            t = time.perf_counter()
            rc = search(ref, None, 0, ptrs[0], ptrs[1], ptrs[2], sp)
            if poll:
                while st_np[0] < 0:
                    pass
            else:
                if not mapped:
                    for h, dvc in zip((opt_h, st_h, plan_h), dbufs):
                        h.copy_(dvc, non_blocking=True)
                hip.hipStreamSynchronize(sp)
            if it >= 10:
                lat.append((time.perf_counter() - t) * 1e6)
            if rc != 0:
                raise RuntimeError(f"cfp_search_chain returned {rc}")
        hip.hipStreamSynchronize(sp)
        return lat

    sync_lat = run(False, 200)
    poll_lat = run(True, 200) if mapped else sync_lat
    rec = {"workload": "chain_gpt_n24_k16", "median": float(np.median(poll_lat)),
           "p10": float(np.percentile(poll_lat, 10)), "p90": float(np.percentile(poll_lat, 90)),
           "median_stream_sync": float(np.median(sync_lat)), "calls": len(poll_lat),
           "form": ("cfp_search_chain, one launch, outputs in mapped pinned host memory; median: the host polls "
                    "the status word; median_stream_sync: hipStreamSynchronize") if mapped
           else "cfp_search_chain, one launch, outputs copied back to pinned host memory, stream synchronised"}
    return rec, (opt_h.numpy().copy(), plan_h.numpy().copy(), st_h.numpy().copy())


COPY_BYTES = 512 << 20


def calibrate_copy() -> int:
    """A plain copy of COPY_BYTES bytes, three times: rocprofv3's FETCH_SIZE and
    WRITE_SIZE of this dispatch give the counter-to-byte scale factors."""
    import torch

    a = torch.ones(COPY_BYTES // 4, dtype=torch.int32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": COPY_BYTES, "copy_bytes_written": COPY_BYTES, "copies": 3}), flush=True)
    return 0


def host_info() -> dict:
    """CPU model and core counts of the host the baseline runs on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    return {"cpu_model": model, "logical_cpus": os.cpu_count() or 1, "cpus_available": avail}


def measure(name: str, steps: int, warmup: int, cpu_s: float, frontier: bool = False,
            chain: bool = False) -> dict:
    """Time `steps` whole passes (forward + traceback) of one workload and
    return its record: step time, cells/s in the metric's unit, the dominant
    kernel's and the forward call's roofline fractions, and, in the CPU leg
    (cpu_s > 0), parity of this run's results against the oracle on the full
    workload and the oracle's rate on the host cores (without the leg, parity
    is reported as null: not checked)."""
    import dataclasses

    import torch

    from workloads import configs

    cfg = configs.BY_NAME[name]
    data = configs.make(cfg)
    if chain:
        if cfg.form != "scan":
            raise SystemExit("--chain applies to the scan workload")
        cfg = dataclasses.replace(cfg, form="chain")
    if frontier:
        if cfg.form != "mem":
            raise SystemExit("--frontier applies to the memory workload")
        data = dict(data, budget=np.full(cfg.B, cfg.M - 1, np.int32))  # the pass covers every budget
    r = Runner(cfg, data, frontier=frontier)
    for _ in range(warmup):
        r.forward()
        r.traceback()
    torch.cuda.synchronize()

    # Timed region: K whole steps (forward + traceback) with nothing else on the
    # stream; an event record costs several microseconds of GPU time, so the
    # per-phase split and the kernel timer come from further, instrumented passes.
    t0 = time.perf_counter()
    for _ in range(steps):
        r.forward()
        r.traceback()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # The library brackets each launch of the dominant kernel with HIP events
    # attached to its dispatch, on the stream it is launched on.  The timer is
    # armed for one step at a time (128 events; cfp_timer_stop waits for them):
    # armed once for all the steps, with thousands of fresh events, some timed
    # launches showed millisecond stalls that neither the kernel trace nor a
    # per-step timer ever shows.
    L = r.L
    kern_ms, kern_launches = 0.0, 0
    for _ in range(steps):
        L.cfp_timer_start(64)
        r.forward()
        r.traceback()
        ms, n = L.cfp_timer_stop()
        kern_ms += ms
        kern_launches += n
    # The forward call and the traceback by stream events, the timer off.
    # Medians: an interval that opens while the GPU has caught up with the host
    # also holds any host stall before the next launch (milliseconds, now and then).
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    for a, m, b in ev:
        a.record(r.stream)
        r.forward()
        m.record(r.stream)
        r.traceback()
        b.record(r.stream)
    torch.cuda.synchronize()
    fwd_ms = float(np.median([a.elapsed_time(m) for a, m, _ in ev]))
    tb_ms = float(np.median([m.elapsed_time(b) for _, m, b in ev]))
    ms_per_step = wall * 1e3 / steps

    cells = cells_of(cfg, data)
    value = cells / (ms_per_step * 1e-3)
    work = scan_gemm_cells(cfg) if cfg.form == "scan" else cells
    # per launch: the algorithmic cells of one launch over its average duration
    # (the scan's products differ in size per level: total cells over total time)
    kern_avg_ms = kern_ms / max(kern_launches, 1)
    kern_cells_s = work * steps / (kern_ms * 1e-3) if kern_launches else 0.0
    fwd_cells_s = work / (fwd_ms * 1e-3)

    gpu_out = {"opt": r.frontier[:, -1].cpu().numpy() if frontier else r.opt.cpu().numpy(),
               "plan": r.plan.cpu().numpy(), "status": r.status.cpu().numpy(),
               "frontier": r.frontier.cpu().numpy() if frontier else None}

    wl = {"workload": cfg.name, "blocks": cfg.N, "strategies": cfg.K, "searches": cfg.B, "resharding_tables": 12}
    if chain:
        wl["form"] = "chain search (cfp_dp_chain, chunk-parallel), not the scan"
    if cfg.form == "seg":
        wl = {"workload": cfg.name, "segments": cfg.N, "plans": cfg.K, "searches": cfg.B,
              "boundary_tables": "2 x 3 x 3", "blocks_per_segment": 4, "strategies_per_block": 3}
    if cfg.form == "mem":
        wl.update({"memory_buckets": cfg.M, "budgets": "every budget 0..M-1" if frontier else "1023-32b"})
    mode = "frontier" if frontier else "chain" if chain else ""
    kernel = KERNELS[cfg.name + ":chain" if chain else cfg.name][0]
    rec = {
        "config": wl,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_per_step,
        "value": value,
        "unit": "cell/s",
        "forward_ms": fwd_ms,
        "traceback_ms": tb_ms,
        "parity_vs_oracle": None,
        "roofline": {"bound": "alu", "achieved": kern_cells_s / 1e12, "peak": PEAK_CELLS / 1e12, "unit": "Tcell/s",
                     "frac": kern_cells_s / PEAK_CELLS,
                     "traffic": traffic_bytes(cfg.name, mode),
                     "kernel": kernel,
                     "kernel_role": KERNEL_ROLE.get(cfg.name + ":chain" if chain else cfg.name, "the forward pass"),
                     "kernel_launches_per_step": kern_launches / steps,
                     "kernel_avg_us": kern_avg_ms * 1e3,
                     "forward_call_cells_per_s": fwd_cells_s,
                     "forward_call_frac": fwd_cells_s / PEAK_CELLS,
                     "step_frac": (work / (ms_per_step * 1e-3)) / PEAK_CELLS},
    }
    if cfg.form == "scan":
        rec["roofline"]["cells_counted"] = ("min-plus matrix-product cells (N-1)*K^3 per search; value counts "
                                            "K^2 per block per search")
        rec["scan_gemm_cells_per_s"] = work / (ms_per_step * 1e-3)
    if cfg.form == "seg":
        rec["roofline"]["cells_counted"] = ("chain-equivalent K^2 per segment step; the factorised step does "
                                            "K + L*F work, so the fraction is not a VALU utilisation")
    lat_out = None
    if cfg.N <= 64 and cfg.B == 1:
        rec["search_latency_us"], lat_out = search_latency_us(r.stream)
    if cpu_s > 0:
        # the CPU leg: the oracle's answers for the GPU results of this run, then its timing
        rec["parity_vs_oracle"] = oracle_parity(cfg, data, gpu_out)
        if lat_out is not None:
            rec["search_latency_us"]["parity_vs_oracle"] = oracle_parity(
                cfg, data, {"opt": lat_out[0], "plan": lat_out[1], "status": lat_out[2], "frontier": None})
        rec["cpu_baseline"] = cpu_baseline(cfg, data, budget_s=cpu_s)
    del r
    torch.cuda.empty_cache()
    return rec


# Records of the default run, in order; the headline is the largest workload.
ALL_RUNS = [("chain_gpt_n24_k16", {}), ("chain_gpt_n1152_k64", {}), ("mem_llama_n288_k32", {}),
            ("mem_llama_n288_k32", {"frontier": True}), ("chain_wide_n512_k256", {}),
            ("scan_n4096_k512", {}), ("scan_n4096_k512", {"chain": True}), ("seg_gpt_n96_k81", {})]
HEADLINE = "scan_n4096_k512"


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default=None,
                    help="time one workload only (default: every workload, headline on the largest)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=None,
                    help="seconds of oracle work per CPU baseline (default 12 for the headline, 4 for the others)")
    ap.add_argument("--chain", action="store_true",
                    help="scan workload only: run the chain search (cfp_dp_chain) instead of the min-plus scan")
    ap.add_argument("--frontier", action="store_true",
                    help="memory workload only: time the budget frontier (every budget 0..M-1 in one pass)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 512 MiB device-to-device copy (reference for the HBM byte counters)")
    args = ap.parse_args()
    if args.calibrate_copy:
        return calibrate_copy()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the searches of a batch are independent, so a run on several GPUs "
              "would only split the batch; no multi-GPU path is built.", file=sys.stderr)
        return 2

    base = {"metric": METRIC, "n_gpus": 1, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "u32", "data": "synthetic"}
    if args.config is not None:
        cpu_s = 0.0 if args.no_cpu else (args.cpu_seconds or 10.0)
        rec = measure(args.config, args.steps, args.warmup, cpu_s, frontier=args.frontier,
                      chain=args.chain)
        if "cpu_baseline" in rec:
            rec["cpu_baseline"]["host"] = host_info()
        out = dict(base, **rec)
        print(json.dumps(out), flush=True)
        return 0 if rec["parity_vs_oracle"] is not False else 1

    records = {}
    for name, kw in ALL_RUNS:
        key = name + "".join(":" + k for k in sorted(kw))
        head = key == HEADLINE
        cpu_s = 0.0 if args.no_cpu else (args.cpu_seconds or (12.0 if head else 4.0))
        print(f"bench: {key}", file=sys.stderr, flush=True)
        records[key] = measure(name, args.steps, args.warmup, cpu_s, **kw)
    head = records[HEADLINE]
    out = dict(base)
    for k in ("value", "unit", "steps", "warmup", "ms_per_step", "config", "forward_ms", "traceback_ms",
              "parity_vs_oracle", "roofline", "scan_gemm_cells_per_s", "cpu_baseline"):
        if k in head:
            out[k] = head[k]
    out["config"] = dict(head["config"], note="largest workload; every workload is in `configs`")
    if "cpu_baseline" in out:
        out["cpu_baseline"] = dict(out["cpu_baseline"], host=host_info())
    out["search_latency_us"] = records["chain_gpt_n24_k16"].get("search_latency_us")
    out["parity_all"] = all(r["parity_vs_oracle"] is not False for r in records.values())
    out["configs"] = records
    print(json.dumps(out), flush=True)
    return 0 if out["parity_all"] else 1


if __name__ == "__main__":
    sys.exit(main())
