"""Seeded synthetic inputs for the chain DP (cost tables, resharding tables,
memory tables, budgets).

This module holds no arithmetic of the search itself: it only draws the
integer tables that stand in for the profiled quantities of the paper's cost
model (per-block time p_n + c_n, resharding time r_n, peak memory m_n; Sec. 4.2
and 4.4, Eq. T and Eq. M).  Both the CPU oracle and the GPU library are fed
the arrays produced here.

Generator: a counter-based stream.  Element k of stream (seed, tag) is

    u_k = mix64((seed XOR tag*PHI) + (k+1)*PHI  mod 2^64)

where mix64 is the SplitMix64 output finaliser (Steele, Lea and Flood,
"Fast splittable pseudorandom number generators", OOPSLA 2014) and PHI is its
golden-ratio increment.  A uniform integer in [lo, hi) is
lo + (((u_k >> 32) * (hi - lo)) >> 32).

Tags and element orders:
    TAG_COST = 1   cost[b][i][s]   k = (b*N + i)*K + s
    TAG_R    = 2   rtab[e][t][s]   k = (e*K + t)*K + s   (diagonal set to 0)
    TAG_ZERO = 3   per table, the off-diagonal entries are ranked by
                   (u_k, flat index) and the smallest `zeros` are set to 0
    TAG_MEM  = 4   mem[b][i][s]    k = (b*N + i)*K + s
    TAG_RB   = 5   rbound[e][l][f] k = (e*S + l)*S + f     (l == f set to 0)
"""
from __future__ import annotations

import numpy as np

PHI = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

TAG_COST = 1
TAG_R = 2
TAG_ZERO = 3
TAG_MEM = 4
TAG_RB = 5

COST_INF = 0x7FFFFFFF  # "strategy unavailable" marker in a cost table


def mix64(z: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser on a uint64 array (wrapping arithmetic, in place)."""
    t = np.empty_like(z)
    np.right_shift(z, np.uint64(30), out=t)
    np.bitwise_xor(z, t, out=z)
    np.multiply(z, _M1, out=z)
    np.right_shift(z, np.uint64(27), out=t)
    np.bitwise_xor(z, t, out=z)
    np.multiply(z, _M2, out=z)
    np.right_shift(z, np.uint64(31), out=t)
    np.bitwise_xor(z, t, out=z)
    return z


def stream(seed: int, tag: int, start: int, count: int) -> np.ndarray:
    """Elements start .. start+count-1 of stream (seed, tag) as uint64."""
    with np.errstate(over="ignore"):
        base = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) ^ (np.uint64(tag) * PHI)
        z = np.arange(start + 1, start + count + 1, dtype=np.uint64)
        np.multiply(z, PHI, out=z)
        np.add(z, base, out=z)
    return mix64(z)


def uniform_int(u: np.ndarray, lo: int, hi: int) -> np.ndarray:
    """Map uint64 draws to integers in [lo, hi) (multiply-shift, no modulo).
    Overwrites u."""
    if hi <= lo:
        raise ValueError("empty range")
    np.right_shift(u, np.uint64(32), out=u)
    np.multiply(u, np.uint64(hi - lo), out=u)
    np.right_shift(u, np.uint64(32), out=u)
    return u.view(np.int64) + lo


def make_cost(seed: int, B: int, N: int, K: int, lo: int, hi: int) -> np.ndarray:
    u = stream(seed, TAG_COST, 0, B * N * K)
    return uniform_int(u, lo, hi).astype(np.int32).reshape(B, N, K)


def make_rtab(seed: int, E: int, K: int, lo: int, hi: int, zeros: int = 0) -> np.ndarray:
    """E resharding tables rtab[e][t][s]: t = strategy of the earlier block,
    s = strategy of the later one.  Diagonal 0 (no resharding when both
    blocks keep the same strategy); `zeros` further off-diagonal entries per
    table set to 0 (communication-free pairs)."""
    u = stream(seed, TAG_R, 0, E * K * K)
    r = uniform_int(u, lo, hi).astype(np.int32).reshape(E, K, K)
    idx = np.arange(K)
    r[:, idx, idx] = 0
    if zeros:
        if zeros > K * (K - 1):
            raise ValueError("more zeros than off-diagonal entries")
        uz = stream(seed, TAG_ZERO, 0, E * K * K).reshape(E, K * K)
        flat = np.arange(K * K, dtype=np.int64)
        offdiag = (flat // K) != (flat % K)
        for e in range(E):
            cand = flat[offdiag]
            order = np.lexsort((cand, uz[e, cand]))  # primary key u, then index
            chosen = cand[order[:zeros]]
            r[e].reshape(-1)[chosen] = 0
    return r


def make_mem(seed: int, B: int, N: int, K: int, lo: int, hi: int) -> np.ndarray:
    u = stream(seed, TAG_MEM, 0, B * N * K)
    return uniform_int(u, lo, hi).astype(np.uint8).reshape(B, N, K)


def make_rbound(seed: int, E: int, S: int, lo: int, hi: int) -> np.ndarray:
    """Boundary resharding tables [E][S][S] (last block strategy -> first
    block strategy), uniform in [lo, hi), zero where the strategies match."""
    u = stream(seed, TAG_RB, 0, E * S * S)
    r = uniform_int(u, lo, hi).astype(np.int32).reshape(E, S, S)
    r[:, np.arange(S), np.arange(S)] = 0
    return r


def digit_maps(P: int, S: int) -> tuple[np.ndarray, np.ndarray]:
    """Plan t = sum_j x_j S^j of a segment of P blocks with S strategies each:
    (last[t], first[t]) = (x_{P-1}, x_0)."""
    t = np.arange(S ** P)
    return (t // S ** (P - 1)).astype(np.uint8), (t % S).astype(np.uint8)


def periodic_redge(N: int, E: int) -> np.ndarray:
    """Edge (i-1 -> i) uses table i mod E; entry 0 is unused (block 0 has no
    incoming edge).  Table 0 is therefore the edge that crosses from one
    layer of E blocks into the next."""
    return (np.arange(N, dtype=np.int64) % E).astype(np.int32)


def make_chain(seed: int, N: int, K: int, B: int, E: int = 12,
               c_range=(10_000, 1_000_000), r_range=(10_000, 1_000_000),
               zeros: int = 0) -> dict:
    return {
        "cost": make_cost(seed, B, N, K, *c_range),
        "rtab": make_rtab(seed, E, K, *r_range, zeros=zeros),
        "redge": periodic_redge(N, E),
    }
