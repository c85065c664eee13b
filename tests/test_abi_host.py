"""The C ABI on the CPU: the library loads, exports every function that
include/cfp.h declares, and rejects bad arguments synchronously without
touching a device (no GPU is needed for any of these)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2504_00598_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "cfp.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cfp_[a-z_]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(L.EXPORTED)


def test_every_declared_symbol_is_exported():
    lib = L.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_only_the_abi_is_exported():
    import subprocess
    out = subprocess.check_output(["nm", "-D", "--defined-only", L.LIB_PATH], text=True)
    names = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    assert names == set(L.EXPORTED)


def test_r_limit_values():
    # packed (value, index) words: b = max(4, ceil(log2 K)) index bits
    assert L.cfp_r_limit(L.CFP_V_CHAIN, 16) == 2 ** 26
    assert L.cfp_r_limit(L.CFP_V_CHAIN, 64) == 2 ** 24
    assert L.cfp_r_limit(L.CFP_V_CHAIN, 65) == 2 ** 25 - 1
    assert L.cfp_r_limit(L.CFP_V_CHAIN, 256) == 2 ** 24 - 1
    assert L.cfp_r_limit(L.CFP_V_CHAIN, 512) == 2 ** 23 - 1
    assert L.cfp_r_limit(L.CFP_V_CHAIN, 513) == 0
    assert L.cfp_r_limit(L.CFP_V_CHAIN, 0) == 0
    assert L.cfp_r_limit(L.CFP_V_MEM, 32) == 2 ** 26
    assert L.cfp_r_limit(L.CFP_V_MEM, 16) == 2 ** 26
    assert L.cfp_r_limit(L.CFP_V_MEM, 64) == 2 ** 25
    assert L.cfp_r_limit(L.CFP_V_MEM, 81) == 2 ** 24
    assert L.cfp_r_limit(L.CFP_V_MEM, 256) == 2 ** 23
    assert L.cfp_r_limit(L.CFP_V_MEM, 257) == 0
    assert L.cfp_r_limit(7, 32) == 0
    # the five workloads' resharding ranges fit their limits
    assert 10_000_000 < L.cfp_r_limit(L.CFP_V_CHAIN, 64)
    assert 10_000_000 < L.cfp_r_limit(L.CFP_V_CHAIN, 256)
    assert 1_000_000 < L.cfp_r_limit(L.CFP_V_MEM, 32)
    assert 1_000_000 < L.cfp_r_limit(L.CFP_V_SCAN, 512)


class HostDesc:
    """A descriptor over host buffers: only ever passed to calls that must
    reject it before any device work."""

    def __init__(self, N=8, K=4, B=2, E=3, redge=None):
        self.cost = np.zeros((B, N, K), np.int32)
        self.rtab = np.zeros((E, K, K), np.int32)
        self.redge = np.zeros(N, np.int32) if redge is None else np.asarray(redge, np.int32)
        self.c = L.cfp_chain_desc(N, K, B, E, self.cost.ctypes.data, self.rtab.ctypes.data, self.redge.ctypes.data)
        self.buf = np.zeros(64, np.int64)

    @property
    def ref(self):
        return ctypes.byref(self.c)


def call_chain(d, ws_bytes=None, ws=True, opt=True):
    lib = L.lib()
    p = d.buf.ctypes.data
    need = lib.cfp_workspace_bytes(d.ref, L.CFP_V_CHAIN, 0)
    return lib.cfp_dp_chain(d.ref, p if ws else None, need - 1 if ws_bytes is None else ws_bytes,
                            p if opt else None, p, None)


def test_workspace_sizes():
    lib = L.lib()
    d = HostDesc(N=1152, K=64, B=256)
    chain = lib.cfp_workspace_bytes(d.ref, L.CFP_V_CHAIN, 0)
    assert chain >= 256 * 1152 * 64  # one argmin byte per (search, block, state)
    assert lib.cfp_workspace_bytes(d.ref, L.CFP_V_MEM, 1024) > 0   # memory variant: K <= 256, any tables
    wide = HostDesc(N=10, K=257, B=2)
    assert lib.cfp_workspace_bytes(wide.ref, L.CFP_V_MEM, 64) == 0  # beyond the memory variant's K
    dm = HostDesc(N=288, K=32, B=16)
    mem = lib.cfp_workspace_bytes(dm.ref, L.CFP_V_MEM, 1024)
    assert mem >= 16 * 288 * 32 * 1024  # one argmin byte per (search, block, state, bucket)
    assert lib.cfp_workspace_bytes(dm.ref, L.CFP_V_MEM, 0) == 0
    assert lib.cfp_workspace_bytes(d.ref, 9, 0) == 0
    d.c.k = 513
    assert lib.cfp_workspace_bytes(d.ref, L.CFP_V_CHAIN, 0) == 0
    assert lib.cfp_workspace_bytes(None, L.CFP_V_CHAIN, 0) == 0


@pytest.mark.parametrize("field,value,code", [
    ("n_blocks", 0, L.CFP_ERR_ARG),
    ("k", 0, L.CFP_ERR_ARG),
    ("k", 513, L.CFP_ERR_UNSUPPORTED),
    ("batch", 0, L.CFP_ERR_ARG),
    ("n_tables", 0, L.CFP_ERR_ARG),
    ("cost", None, L.CFP_ERR_ARG),
    ("rtab", None, L.CFP_ERR_ARG),
    ("redge", None, L.CFP_ERR_ARG),
])
def test_descriptor_errors(field, value, code):
    d = HostDesc()
    setattr(d.c, field, value)
    assert call_chain(d) == code


def test_redge_out_of_range():
    d = HostDesc(N=5, E=3, redge=[99, 0, 1, 3, 2])  # redge[0] is ignored, redge[3] = 3 is not
    assert call_chain(d) == L.CFP_ERR_RANGE
    d = HostDesc(N=5, E=3, redge=[0, 0, -1, 0, 0])
    assert call_chain(d) == L.CFP_ERR_RANGE


def test_workspace_too_small_and_nulls():
    d = HostDesc()
    assert call_chain(d) == L.CFP_ERR_WORKSPACE          # one byte short
    assert call_chain(d, ws=False, ws_bytes=1 << 30) == L.CFP_ERR_WORKSPACE
    assert call_chain(d, opt=False, ws_bytes=1 << 30) == L.CFP_ERR_ARG


def test_other_entry_points_validate():
    lib = L.lib()
    d = HostDesc()
    p = d.buf.ctypes.data
    assert lib.cfp_dp_chain_mem(d.ref, None, 16, p, p, 1 << 30, p, p, None) == L.CFP_ERR_ARG
    assert lib.cfp_dp_chain_mem(d.ref, p, 0, p, p, 1 << 30, p, p, None) == L.CFP_ERR_ARG
    assert lib.cfp_dp_chain_mem(d.ref, p, 5000, p, p, 1 << 30, p, p, None) == L.CFP_ERR_UNSUPPORTED
    assert lib.cfp_dp_chain_mem(d.ref, p, 16, p, p, 10, p, p, None) == L.CFP_ERR_WORKSPACE
    assert lib.cfp_minplus_scan(d.ref, p, 10, p, p, None) == L.CFP_ERR_WORKSPACE
    assert lib.cfp_traceback(d.ref, L.CFP_V_CHAIN, 0, p, 10, p, None) == L.CFP_ERR_WORKSPACE
    assert lib.cfp_traceback(d.ref, 7, 0, p, 1 << 30, p, None) == L.CFP_ERR_ARG
    assert lib.cfp_traceback(d.ref, L.CFP_V_CHAIN, 0, p, 1 << 30, None, None) == L.CFP_ERR_ARG


def test_status_strings():
    for code in (0, 1, 2, 3, 4, -1, -2, -3, -4, -5):
        assert L.status_string(code) != "unknown code"
    assert L.status_string(12345) == "unknown code"
