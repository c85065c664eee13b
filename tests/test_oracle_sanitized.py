"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer runs
the pin battery cleanly: no out-of-bounds access, use after free, signed
overflow or other undefined behaviour on the inputs the pins use (tiny chains
with ties, unavailable strategies, memory budgets, the frontier).

The sanitized copy is built in a temporary directory with gcc on the CPU and
loaded into a child Python process with the sanitizer runtime preloaded; the
oracle's own build is not touched."""
from __future__ import annotations

import os
import subprocess
import sys
import textwrap

import pytest

from oracle import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_clean_under_asan_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc has no AddressSanitizer runtime here")
    so = tmp_path / "liboracle_san.so"
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-shared", "-fPIC", "-pthread",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                           O.SRC, "-o", str(so)])
    script = textwrap.dedent(f"""
        import ctypes, sys
        import numpy as np
        sys.path.insert(0, {ROOT!r})
        from oracle import oracle as O
        real = O.lib()
        L = ctypes.CDLL({str(so)!r})
        for fn in ("oracle_chain", "oracle_chain_mem", "oracle_mem_frontier", "oracle_chain_values",
                   "oracle_plan_cost", "oracle_plan_mem"):
            getattr(L, fn).argtypes = getattr(real, fn).argtypes
            getattr(L, fn).restype = getattr(real, fn).restype
        O._lib = L
        from tests.test_oracle_mutants import pins_pass
        assert pins_pass(), "pin battery failed on the sanitized oracle"
        rs = np.random.default_rng(5)
        B, N, K = 3, 40, 7
        cost = rs.integers(0, 2**31 - 1, size=(B, N, K)).astype(np.int32)
        cost[0, 5, :] = 0x7FFFFFFF
        rtab = rs.integers(0, 2**30, size=(4, K, K)).astype(np.int32)
        redge = rs.integers(0, 4, size=N).astype(np.int32)
        mem = rs.integers(0, 9, size=(B, N, K)).astype(np.uint8)
        O.chain(cost, rtab, redge, nthreads=3)
        O.chain_mem(cost, rtab, redge, mem, np.array([0, 100, 300], np.int32), nthreads=3)
        O.mem_frontier(cost, rtab, redge, mem, 64, nthreads=3)
        print("sanitized oracle ok")
    """)
    env = dict(os.environ)
    env["LD_PRELOAD"] = asan
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([sys.executable, "-c", script], capture_output=True, text=True, env=env, cwd=ROOT,
                       timeout=600)
    assert r.returncode == 0 and "sanitized oracle ok" in r.stdout, r.stdout[-3000:] + r.stderr[-3000:]
