"""ctypes binding of libcfp.so.

Argument marshalling only: every step of the search runs in the HIP kernels
behind the C ABI (include/cfp.h).  torch supplies device memory and the
current stream.  If libcfp.so is missing the import-time load raises; there is
no other code path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcfp.so")

# Synchronous return codes and device statuses (values of include/cfp.h).
CFP_OK = 0
CFP_ERR_ARG = -1
CFP_ERR_RANGE = -2
CFP_ERR_WORKSPACE = -3
CFP_ERR_UNSUPPORTED = -4
CFP_ERR_HIP = -5
CFP_ST_OK = 0
CFP_ST_INFEASIBLE = 1
CFP_ST_OVERFLOW = 2
CFP_ST_TIMEOUT = 3
CFP_ST_BADINPUT = 4
CFP_V_CHAIN = 0
CFP_V_MEM = 1
CFP_V_SCAN = 2
CFP_V_SEG = 3
CFP_COST_INF = 0x7FFFFFFF
CFP_MAX_K = 512

EXPORTED = ("cfp_r_limit", "cfp_workspace_bytes", "cfp_dp_chain", "cfp_dp_chain_mem", "cfp_mem_frontier",
            "cfp_minplus_scan", "cfp_traceback", "cfp_segment_workspace_bytes", "cfp_dp_segments",
            "cfp_traceback_segments", "cfp_status_string", "cfp_timer_start", "cfp_timer_stop",
            "cfp_search_chain", "cfp_search_chain_noalloc")


class CfpError(RuntimeError):
    def __init__(self, fn: str, code: int):
        self.code = code
        super().__init__(f"{fn} failed: {code} ({status_string(code)})")


class cfp_chain_desc(ctypes.Structure):
    _fields_ = [
        ("n_blocks", ctypes.c_int32),
        ("k", ctypes.c_int32),
        ("batch", ctypes.c_int32),
        ("n_tables", ctypes.c_int32),
        ("cost", ctypes.c_void_p),
        ("rtab", ctypes.c_void_p),
        ("redge", ctypes.c_void_p),
    ]


class cfp_segment_desc(ctypes.Structure):
    _fields_ = [
        ("n_segments", ctypes.c_int32),
        ("k", ctypes.c_int32),
        ("batch", ctypes.c_int32),
        ("n_tables", ctypes.c_int32),
        ("n_last", ctypes.c_int32),
        ("n_first", ctypes.c_int32),
        ("cost", ctypes.c_void_p),
        ("rbound", ctypes.c_void_p),
        ("last", ctypes.c_void_p),
        ("first", ctypes.c_void_p),
        ("redge", ctypes.c_void_p),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libcfp.so (raises OSError if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise OSError(f"{LIB_PATH} is missing: build it with `python -m paper_2504_00598_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I32 = ctypes.c_void_p, ctypes.c_int32
        D = ctypes.POINTER(cfp_chain_desc)
        L.cfp_r_limit.argtypes = [I32, I32]
        L.cfp_r_limit.restype = I32
        L.cfp_workspace_bytes.argtypes = [D, I32, I32]
        L.cfp_workspace_bytes.restype = ctypes.c_size_t
        L.cfp_dp_chain.argtypes = [D, P, ctypes.c_size_t, P, P, P]
        L.cfp_dp_chain.restype = ctypes.c_int
        L.cfp_dp_chain_mem.argtypes = [D, P, I32, P, P, ctypes.c_size_t, P, P, P]
        L.cfp_dp_chain_mem.restype = ctypes.c_int
        L.cfp_mem_frontier.argtypes = [D, P, I32, P, ctypes.c_size_t, P, P, P]
        L.cfp_mem_frontier.restype = ctypes.c_int
        L.cfp_minplus_scan.argtypes = [D, P, ctypes.c_size_t, P, P, P]
        L.cfp_minplus_scan.restype = ctypes.c_int
        L.cfp_traceback.argtypes = [D, I32, I32, P, ctypes.c_size_t, P, P]
        L.cfp_traceback.restype = ctypes.c_int
        SD = ctypes.POINTER(cfp_segment_desc)
        L.cfp_segment_workspace_bytes.argtypes = [SD]
        L.cfp_segment_workspace_bytes.restype = ctypes.c_size_t
        L.cfp_dp_segments.argtypes = [SD, P, ctypes.c_size_t, P, P, P]
        L.cfp_dp_segments.restype = ctypes.c_int
        L.cfp_traceback_segments.argtypes = [SD, P, ctypes.c_size_t, P, P]
        L.cfp_traceback_segments.restype = ctypes.c_int
        L.cfp_search_chain.argtypes = [D, P, ctypes.c_size_t, P, P, P, P]
        L.cfp_search_chain.restype = ctypes.c_int
        L.cfp_search_chain_noalloc.argtypes = [D, P, P, P, P]
        L.cfp_search_chain_noalloc.restype = ctypes.c_int
        L.cfp_timer_start.argtypes = [I32]
        L.cfp_timer_start.restype = ctypes.c_int
        L.cfp_timer_stop.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I32)]
        L.cfp_timer_stop.restype = ctypes.c_int
        L.cfp_status_string.argtypes = [ctypes.c_int]
        L.cfp_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().cfp_status_string(int(code)).decode()


def cfp_r_limit(variant: int, k: int) -> int:
    return int(lib().cfp_r_limit(variant, k))


def cfp_timer_start(max_launches: int) -> None:
    rc = lib().cfp_timer_start(int(max_launches))
    if rc != CFP_OK:
        raise CfpError("cfp_timer_start", rc)


def cfp_timer_stop() -> tuple[float, int]:
    """(summed device milliseconds, bracketed launches) of the armed timer."""
    ms, n = ctypes.c_double(0.0), ctypes.c_int32(0)
    rc = lib().cfp_timer_stop(ctypes.byref(ms), ctypes.byref(n))
    if rc != CFP_OK:
        raise CfpError("cfp_timer_stop", rc)
    return ms.value, n.value


# ------------------------------------------------------------- marshalling --

def _ptr(t) -> int | None:
    """Device address of a torch tensor (or None)."""
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream) -> int | None:
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


class Desc:
    """A cfp_chain_desc plus the objects that keep its memory alive."""

    def __init__(self, cost, rtab, redge):
        import torch

        if not (isinstance(cost, torch.Tensor) and isinstance(rtab, torch.Tensor)):
            raise TypeError("cost and rtab must be torch tensors on the GPU")
        if cost.dtype != torch.int32 or rtab.dtype != torch.int32:
            raise TypeError("cost and rtab must be int32")
        if not (cost.is_cuda and rtab.is_cuda):
            raise TypeError("cost and rtab must be device tensors")
        if not (cost.is_contiguous() and rtab.is_contiguous()):
            raise ValueError("cost and rtab must be contiguous")
        if cost.dim() != 3 or rtab.dim() != 3:
            raise ValueError("cost is [B][N][K] and rtab is [E][K][K]")
        B, N, K = cost.shape
        self.redge = np.ascontiguousarray(np.asarray(redge, dtype=np.int32))
        if self.redge.shape != (N,):
            raise ValueError("redge must have N entries")
        self.cost, self.rtab = cost, rtab
        self.B, self.N, self.K, self.E = int(B), int(N), int(K), int(rtab.shape[0])
        self.c = cfp_chain_desc(self.N, self.K, self.B, self.E, _ptr(cost), _ptr(rtab),
                                self.redge.ctypes.data_as(ctypes.c_void_p).value)

    @property
    def ref(self):
        return ctypes.byref(self.c)


class SegDesc:
    """A cfp_segment_desc plus the objects that keep its memory alive.  cost
    [B][N][K] int32, rbound [E][L][F] int32, last/first [K] uint8 are device
    tensors; redge [N] is host data."""

    def __init__(self, cost, rbound, last, first, redge):
        import torch

        for name, t, dt in (("cost", cost, torch.int32), ("rbound", rbound, torch.int32),
                            ("last", last, torch.uint8), ("first", first, torch.uint8)):
            if not isinstance(t, torch.Tensor) or t.dtype != dt or not t.is_cuda or not t.is_contiguous():
                raise TypeError(f"{name} must be a contiguous {dt} device tensor")
        if cost.dim() != 3 or rbound.dim() != 3:
            raise ValueError("cost is [B][N][K] and rbound is [E][L][F]")
        B, N, K = cost.shape
        if tuple(last.shape) != (K,) or tuple(first.shape) != (K,):
            raise ValueError("last and first have K entries")
        self.redge = np.ascontiguousarray(np.asarray(redge, dtype=np.int32))
        if self.redge.shape != (N,):
            raise ValueError("redge must have N entries")
        self.cost, self.rbound, self.last, self.first = cost, rbound, last, first
        E, Lc, Fc = rbound.shape
        self.B, self.N, self.K, self.E, self.L, self.F = int(B), int(N), int(K), int(E), int(Lc), int(Fc)
        self.c = cfp_segment_desc(self.N, self.K, self.B, self.E, self.L, self.F, _ptr(cost), _ptr(rbound),
                                  _ptr(last), _ptr(first), self.redge.ctypes.data_as(ctypes.c_void_p).value)

    @property
    def ref(self):
        return ctypes.byref(self.c)


def cfp_segment_workspace_bytes(desc: SegDesc) -> int:
    return int(lib().cfp_segment_workspace_bytes(desc.ref))


def cfp_dp_segments(desc: SegDesc, ws=None, opt=None, status=None, stream=None):
    """Enqueue the segment search.  Returns (opt, status, ws)."""
    import torch

    dev = desc.cost.device
    ws = _alloc(cfp_segment_workspace_bytes(desc), dev) if ws is None else ws
    opt = torch.empty(desc.B, dtype=torch.int64, device=dev) if opt is None else opt
    status = torch.empty(desc.B, dtype=torch.int32, device=dev) if status is None else status
    _check("cfp_dp_segments", lib().cfp_dp_segments(desc.ref, _ptr(ws), ws.numel(), _ptr(opt), _ptr(status),
                                                    _stream(stream)))
    return opt, status, ws


def cfp_traceback_segments(desc: SegDesc, ws, plan=None, stream=None):
    """Enqueue the plan recovery of a segment search.  Returns plan [B][N]."""
    import torch

    plan = torch.empty((desc.B, desc.N), dtype=torch.int32, device=desc.cost.device) if plan is None else plan
    _check("cfp_traceback_segments", lib().cfp_traceback_segments(desc.ref, _ptr(ws), ws.numel(), _ptr(plan),
                                                                  _stream(stream)))
    return plan


CFP_NOALLOC_MAX_BYTES = 32 << 20


def cfp_search_chain(desc: Desc, ws=None, opt=None, status=None, plan=None, stream=None):
    """Enqueue the whole chain search (forward and traceback) in one call; small
    searches run as one kernel launch and need no workspace (ws may be None then,
    and is allocated otherwise).  Returns (opt, status, plan)."""
    import torch

    dev = desc.cost.device
    if ws is None and not chain_search_is_one_launch(desc):
        ws = _alloc(cfp_workspace_bytes(desc, CFP_V_CHAIN), dev)
    opt = torch.empty(desc.B, dtype=torch.int64, device=dev) if opt is None else opt
    status = torch.empty(desc.B, dtype=torch.int32, device=dev) if status is None else status
    plan = torch.empty((desc.B, desc.N), dtype=torch.int32, device=dev) if plan is None else plan
    _check("cfp_search_chain", lib().cfp_search_chain(desc.ref, _ptr(ws) if ws is not None else None,
                                                      ws.numel() if ws is not None else 0, _ptr(opt),
                                                      _ptr(status), _ptr(plan), _stream(stream)))
    return opt, status, plan


def chain_search_is_one_launch(desc: Desc) -> bool:
    """Whether cfp_search_chain runs `desc` as its one-launch path (the rule
    documented in cfp.h)."""
    K, N, B, E = desc.K, desc.N, desc.B, desc.E
    if K > 64 or N > 512 or B > 256 or E > 255:
        return False
    kp = 16 if K <= 16 else 32 if K <= 32 else 64
    return E * kp * (kp + 4) * 4 + N * (5 * kp + 1) <= 61440


def cfp_search_chain_noalloc(desc: Desc, opt=None, status=None, plan=None, stream=None):
    """Enqueue the chain search and its traceback with the workspace in the
    library's static device scratch.  Returns (opt, status, plan)."""
    import torch

    dev = desc.cost.device
    opt = torch.empty(desc.B, dtype=torch.int64, device=dev) if opt is None else opt
    status = torch.empty(desc.B, dtype=torch.int32, device=dev) if status is None else status
    plan = torch.empty((desc.B, desc.N), dtype=torch.int32, device=dev) if plan is None else plan
    _check("cfp_search_chain_noalloc", lib().cfp_search_chain_noalloc(desc.ref, _ptr(opt), _ptr(status), _ptr(plan),
                                                                      _stream(stream)))
    return opt, status, plan


def cfp_workspace_bytes(desc: Desc, variant: int, n_mem: int = 0) -> int:
    return int(lib().cfp_workspace_bytes(desc.ref, variant, n_mem))


def _alloc(nbytes, device):
    import torch

    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _check(fn, rc):
    if rc != CFP_OK:
        raise CfpError(fn, rc)


def cfp_dp_chain(desc: Desc, ws=None, opt=None, status=None, stream=None):
    """Enqueue the unconstrained forward search.  Returns (opt, status, ws)."""
    import torch

    dev = desc.cost.device
    need = cfp_workspace_bytes(desc, CFP_V_CHAIN)
    ws = _alloc(need, dev) if ws is None else ws
    opt = torch.empty(desc.B, dtype=torch.int64, device=dev) if opt is None else opt
    status = torch.empty(desc.B, dtype=torch.int32, device=dev) if status is None else status
    _check("cfp_dp_chain", lib().cfp_dp_chain(desc.ref, _ptr(ws), ws.numel(), _ptr(opt), _ptr(status),
                                              _stream(stream)))
    return opt, status, ws


def cfp_dp_chain_mem(desc: Desc, mem, n_mem: int, budget, ws=None, opt=None, status=None, stream=None):
    """Enqueue the memory-budgeted forward search.  mem [B][N][K] uint8 and
    budget [B] int32 are device tensors.  Returns (opt, status, ws)."""
    import torch

    if mem.dtype != torch.uint8 or budget.dtype != torch.int32 or not (mem.is_cuda and budget.is_cuda):
        raise TypeError("mem must be a uint8 device tensor and budget an int32 device tensor")
    if tuple(mem.shape) != (desc.B, desc.N, desc.K) or tuple(budget.shape) != (desc.B,):
        raise ValueError("mem is [B][N][K] and budget is [B]")
    mem, budget = mem.contiguous(), budget.contiguous()
    dev = desc.cost.device
    need = cfp_workspace_bytes(desc, CFP_V_MEM, n_mem)
    ws = _alloc(need, dev) if ws is None else ws
    opt = torch.empty(desc.B, dtype=torch.int64, device=dev) if opt is None else opt
    status = torch.empty(desc.B, dtype=torch.int32, device=dev) if status is None else status
    _check("cfp_dp_chain_mem", lib().cfp_dp_chain_mem(desc.ref, _ptr(mem), int(n_mem), _ptr(budget), _ptr(ws),
                                                      ws.numel(), _ptr(opt), _ptr(status), _stream(stream)))
    return opt, status, ws


def cfp_mem_frontier(desc: Desc, mem, n_mem: int, ws=None, frontier=None, status=None, stream=None):
    """Enqueue the budget-frontier search.  mem [B][N][K] uint8 is a device
    tensor.  Returns (frontier [B][n_mem] int64, status, ws)."""
    import torch

    if mem.dtype != torch.uint8 or not mem.is_cuda:
        raise TypeError("mem must be a uint8 device tensor")
    if tuple(mem.shape) != (desc.B, desc.N, desc.K):
        raise ValueError("mem is [B][N][K]")
    mem = mem.contiguous()
    dev = desc.cost.device
    need = cfp_workspace_bytes(desc, CFP_V_MEM, n_mem)
    ws = _alloc(need, dev) if ws is None else ws
    frontier = torch.empty((desc.B, int(n_mem)), dtype=torch.int64, device=dev) if frontier is None else frontier
    status = torch.empty(desc.B, dtype=torch.int32, device=dev) if status is None else status
    if tuple(frontier.shape) != (desc.B, int(n_mem)) or frontier.dtype != torch.int64:
        raise ValueError("frontier is [B][n_mem] int64")
    _check("cfp_mem_frontier", lib().cfp_mem_frontier(desc.ref, _ptr(mem), int(n_mem), _ptr(ws), ws.numel(),
                                                      _ptr(frontier), _ptr(status), _stream(stream)))
    return frontier, status, ws


def cfp_minplus_scan(desc: Desc, ws=None, opt=None, status=None, stream=None):
    """Enqueue the min-plus parallel-scan search.  Returns (opt, status, ws)."""
    import torch

    dev = desc.cost.device
    need = cfp_workspace_bytes(desc, CFP_V_SCAN)
    ws = _alloc(need, dev) if ws is None else ws
    opt = torch.empty(desc.B, dtype=torch.int64, device=dev) if opt is None else opt
    status = torch.empty(desc.B, dtype=torch.int32, device=dev) if status is None else status
    _check("cfp_minplus_scan", lib().cfp_minplus_scan(desc.ref, _ptr(ws), ws.numel(), _ptr(opt), _ptr(status),
                                                      _stream(stream)))
    return opt, status, ws


def cfp_traceback(desc: Desc, variant: int, ws, n_mem: int = 0, plan=None, stream=None):
    """Enqueue the plan recovery from a filled workspace.  Returns plan [B][N]."""
    import torch

    plan = torch.empty((desc.B, desc.N), dtype=torch.int32, device=desc.cost.device) if plan is None else plan
    _check("cfp_traceback", lib().cfp_traceback(desc.ref, variant, int(n_mem), _ptr(ws), ws.numel(), _ptr(plan),
                                                _stream(stream)))
    return plan
