"""Oracle of the front-end counts (TEST INFRASTRUCTURE ONLY: imported by the
test suite; the product package never imports it).

profiling_programs follows Sec. 4.3 (Eq. 2) by writing the programs out: one
program per strategy combination of the blocks of each distinct segment, and
one per strategy pair of every pair of blocks joined by a cross-segment
dependency.  Its length is the profiling-space size, counted by enumeration
rather than by the closed form.
"""
from __future__ import annotations

import itertools


def profiling_programs(strategies, deps=()):
    """Every program of the profiling space, as tuples:
    ("segment", i, (s_1, ..., s_K)) and ("reshard", entry, i, j, l, k, s_l, s_k)."""
    programs = []
    for i, seg in enumerate(strategies):
        for combo in itertools.product(*[range(s) for s in seg]):
            programs.append(("segment", i, combo))
    for entry, (i, j, l, k) in enumerate(deps):
        for s_l in range(strategies[i][l]):
            for s_k in range(strategies[j][k]):
                programs.append(("reshard", entry, i, j, l, k, s_l, s_k))
    return programs


def profiling_space_size(strategies, deps=()):
    return len(profiling_programs(strategies, list(deps)))


# ------------------------------------------------------------ Algorithm 1 --
# ParallelBlock grouping (Sec. 3.2, Algorithm 1) with the check of Eq. 1
# evaluated on element-level dependency sets, computed by brute force from
# the operator semantics of Table 1 (row-major reshapes).  Graphs are the
# product's Graph objects (plain data); only shapes and specs are read.

import numpy as np


def _deps_start(shape):
    n = int(np.prod(shape))
    arr = np.empty(n, dtype=object)
    for k in range(n):
        arr[k] = frozenset([k])
    return arr.reshape(shape)


def _deps_apply(deps, op, pos):
    """Dependency sets of op's output elements, given those of operand `pos`."""
    if op.kind == "elementwise":
        return deps
    if op.kind in ("split", "merge"):
        return deps.reshape(op.shape)
    if op.kind == "transpose":
        axes = [0] * len(op.perm)
        for i, j in enumerate(op.perm):
            axes[j] = i
        return np.transpose(deps, axes)
    if op.kind == "broadcast":
        return np.repeat(np.expand_dims(deps, op.axis), op.size, axis=op.axis)
    lhs, out = op.spec.replace(" ", "").split("->")
    mine = lhs.split(",")[pos]
    size = dict(zip(mine, deps.shape))
    red = [c for c in mine if c not in out]
    res = np.empty(op.shape, dtype=object)
    for idx in np.ndindex(*op.shape):
        val = dict(zip(out, idx))
        acc = set()
        for ridx in itertools.product(*[range(size[c]) for c in red]):
            val.update(zip(red, ridx))
            acc |= deps[tuple(val[c] for c in mine)]
        res[idx] = frozenset(acc)
    return res


def preserving(deps, xshape, P):
    """Eq. 1 as a definition: every dimension i of X of size A_i divisible by P
    can be cut into nb blocks (nb divides A_i, nb a multiple of P) that match
    nb contiguous blocks of some dimension j of the current tensor: every
    element's dependencies lie in the X block of its own block number."""
    tshape = deps.shape
    pairs = []
    for a in np.ndindex(*tshape):
        for b in deps[a]:
            pairs.append((a, np.unravel_index(b, xshape)))
    for i, A in enumerate(xshape):
        if A % P:
            continue
        found = False
        for nb in range(P, A + 1, P):
            if A % nb:
                continue
            for j, T in enumerate(tshape):
                if T % nb:
                    continue
                dx, dt = A // nb, T // nb
                if all(b[i] // dx == a[j] // dt for a, b in pairs):
                    found = True
                    break
            if found:
                break
        if not found:
            return False
    return True


def build_parallel_blocks(g, P):
    """Algorithm 1 with the brute-force check: contractions by depth, then
    graph order; each ungrouped one grows a block through its first
    qualifying ungrouped user, depth first."""
    depth = {}
    for o in g.ops.values():
        depth[o.name] = 0 if not o.operands else 1 + max(depth[x] for x in o.operands)
    order = {n: i for i, n in enumerate(g.ops)}
    cons = sorted((o.name for o in g.ops.values() if o.kind == "contraction"), key=lambda n: (depth[n], order[n]))
    grouped, blocks = set(), []
    for s in cons:
        if s in grouped:
            continue
        pb, cur = [s], s
        xshape = g.ops[s].shape
        deps = _deps_start(xshape)
        while True:
            nxt = None
            for u in [o.name for o in g.ops.values() if cur in o.operands]:
                if u in grouped or u in pb:
                    continue
                d2 = _deps_apply(deps, g.ops[u], g.ops[u].operands.index(cur))
                if preserving(d2, xshape, P):
                    nxt, deps = u, d2
                    break
            if nxt is None:
                break
            pb.append(nxt)
            cur = nxt
        grouped.update(pb)
        blocks.append(pb)
    return blocks


def path_preserving(g, path, P):
    deps = _deps_start(g.ops[path[0]].shape)
    for prev, u in zip(path, path[1:]):
        deps = _deps_apply(deps, g.ops[u], g.ops[u].operands.index(prev))
    return preserving(deps, g.ops[path[0]].shape, P)
