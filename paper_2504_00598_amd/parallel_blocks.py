"""ParallelBlock construction, phase 1 (Sec. 3.2, Algorithm 1): grouping the
operators downstream of each tensor contraction while the subgraph stays
parallelism-preserving (Sec. 3.1, Eq. 1), with the element-level dependencies
of Table 1.

A graph is a list of operators in topological order.  Every operator names
its operands and has one output tensor.  Kinds (Table 1):
    "input"        a graph input or parameter (no operands)
    "elementwise"  same shape as its operands; output element a reads element a
    "split"        dimension k of the operand becomes dimensions k, k+1 of
                   sizes (A_k, A_{k+1}); row-major: f_k(a) = A_{k+1} a_k + a_{k+1}
    "merge"        dimensions k, k+1 of the operand become dimension k:
                   f_k(a) = a_k // B_{k+1}, f_{k+1}(a) = a_k mod B_{k+1}
    "transpose"    perm: operand dimension i is output dimension perm[i]
                   (f_i(a) = a_{perm[i]})
    "broadcast"    a new dimension k of size n
    "contraction"  an einsum over its operands; letters of an operand missing
                   from the output are reduced (f_k(a) = every index)

Dependencies are tracked symbolically.  Every dimension of a tensor is a
list of digits (mixed-radix, most significant first), and a digit of the
current tensor either carries a digit of the block's input tensor X (its
index equals that digit's index) or is new (from another operand or a
broadcast); a digit of X that a contraction reduced is free.  A split that
cuts inside a digit refines that digit into two (in X as well); a split that
cannot be expressed on the digits (sizes that do not factor along them)
makes the digits involved opaque.

The check of Eq. 1 (reading): for every dimension i of X whose size is a
multiple of the mesh-axis size P, some positive d_i with (A_i / d_i) a
multiple of P must exist such that partitioning X's dimension i into blocks of
d_i corresponds to partitioning one dimension j of the current tensor into the
same number of blocks, element for element: the leading digits of X's
dimension i, whose sizes multiply to A_i / d_i, lead dimension j of the
current tensor in the same order.  Dimension j may differ from i (reshapes and
transposes move dimensions).

Host-side analysis: no part of it runs on the GPU.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

KINDS = ("input", "elementwise", "split", "merge", "transpose", "broadcast", "contraction")


@dataclass
class Op:
    name: str
    kind: str
    operands: Tuple[str, ...] = ()
    shape: Tuple[int, ...] = ()      # output shape (filled in by Graph.add)
    axis: int = 0                    # split, merge, broadcast
    sizes: Tuple[int, int] = (0, 0)  # split: the two new sizes
    perm: Tuple[int, ...] = ()       # transpose
    size: int = 0                    # broadcast: size of the new dimension
    spec: str = ""                   # contraction: einsum "ab,bc->ac"


class Graph:
    """Operators in insertion (topological) order, with shape inference."""

    def __init__(self):
        self.ops: Dict[str, Op] = {}

    def add(self, op: Op) -> Op:
        if op.name in self.ops:
            raise ValueError(f"duplicate operator {op.name}")
        if op.kind not in KINDS:
            raise ValueError(f"unknown kind {op.kind}")
        for o in op.operands:
            if o not in self.ops:
                raise ValueError(f"{op.name}: operand {o} is not defined before it")
        shapes = [self.ops[o].shape for o in op.operands]
        op.shape = tuple(int(x) for x in _infer_shape(op, shapes))
        self.ops[op.name] = op
        return op

    # convenience constructors
    def input(self, name, shape):
        return self.add(Op(name, "input", shape=tuple(shape)))

    def elementwise(self, name, *operands):
        return self.add(Op(name, "elementwise", tuple(operands)))

    def split(self, name, operand, axis, sizes):
        return self.add(Op(name, "split", (operand,), axis=axis, sizes=tuple(sizes)))

    def merge(self, name, operand, axis):
        return self.add(Op(name, "merge", (operand,), axis=axis))

    def transpose(self, name, operand, perm):
        return self.add(Op(name, "transpose", (operand,), perm=tuple(perm)))

    def broadcast(self, name, operand, axis, size):
        return self.add(Op(name, "broadcast", (operand,), axis=axis, size=size))

    def contraction(self, name, spec, *operands):
        return self.add(Op(name, "contraction", tuple(operands), spec=spec))

    def users(self, name: str) -> List[str]:
        """Operators that read `name`'s output, in graph order."""
        return [o.name for o in self.ops.values() if name in o.operands]

    def depth(self) -> Dict[str, int]:
        """Length of the longest path from a graph input to every operator."""
        d: Dict[str, int] = {}
        for o in self.ops.values():
            d[o.name] = 0 if not o.operands else 1 + max(d[x] for x in o.operands)
        return d


def _parse_spec(spec: str) -> Tuple[List[str], str]:
    lhs, out = spec.replace(" ", "").split("->")
    return lhs.split(","), out


def _infer_shape(op: Op, shapes: Sequence[Tuple[int, ...]]) -> Tuple[int, ...]:
    if op.kind == "input":
        if not op.shape or any(int(x) < 1 for x in op.shape):
            raise ValueError(f"{op.name}: an input needs a positive shape")
        return op.shape
    if op.kind == "elementwise":
        if not shapes or any(s != shapes[0] for s in shapes):
            raise ValueError(f"{op.name}: elementwise operands have one shape")
        return shapes[0]
    (s,) = shapes if op.kind != "contraction" else (None,)
    if op.kind == "split":
        k, (a, b) = op.axis, op.sizes
        if not (0 <= k < len(s)) or a * b != s[k] or a < 1 or b < 1:
            raise ValueError(f"{op.name}: split sizes {op.sizes} do not make dimension {k} of {s}")
        return s[:k] + (a, b) + s[k + 1:]
    if op.kind == "merge":
        k = op.axis
        if not (0 <= k < len(s) - 1):
            raise ValueError(f"{op.name}: cannot merge dimensions {k}, {k + 1} of {s}")
        return s[:k] + (s[k] * s[k + 1],) + s[k + 2:]
    if op.kind == "transpose":
        if sorted(op.perm) != list(range(len(s))):
            raise ValueError(f"{op.name}: {op.perm} is not a permutation of {len(s)} dimensions")
        out = [0] * len(s)
        for i, j in enumerate(op.perm):
            out[j] = s[i]
        return tuple(out)
    if op.kind == "broadcast":
        if not (0 <= op.axis <= len(s)) or op.size < 1:
            raise ValueError(f"{op.name}: bad broadcast")
        return s[:op.axis] + (op.size,) + s[op.axis:]
    # contraction
    ins, out = _parse_spec(op.spec)
    if len(ins) != len(shapes):
        raise ValueError(f"{op.name}: {len(ins)} operands in {op.spec!r}, {len(shapes)} given")
    size: Dict[str, int] = {}
    for letters, sh in zip(ins, shapes):
        if len(letters) != len(sh):
            raise ValueError(f"{op.name}: {letters!r} does not match rank {len(sh)}")
        for c, n in zip(letters, sh):
            if size.setdefault(c, n) != n:
                raise ValueError(f"{op.name}: size of {c!r} disagrees")
    if len(set(out)) != len(out) or any(c not in size for c in out):
        raise ValueError(f"{op.name}: bad output letters {out!r}")
    return tuple(size[c] for c in out)


# ----------------------------------------------------------------- digits --

@dataclass
class _Digit:
    size: int
    x: Optional[int] = None  # the X digit it carries, or None (new)


@dataclass
class _State:
    """Digits of X (per dimension) and of the current tensor T (per dimension)."""
    xdims: List[List[int]]                       # X digit ids, most significant first
    xsize: Dict[int, int]                        # X digit id -> size
    tdims: List[List[_Digit]]
    reduced: set = field(default_factory=set)    # X digits a contraction reduced
    opaque: set = field(default_factory=set)     # X digits no longer expressible
    next_id: int = 0

    @staticmethod
    def start(shape: Sequence[int]) -> "_State":
        st = _State([], {}, [])
        for n in shape:
            xid = st.next_id
            st.next_id += 1
            st.xsize[xid] = int(n)
            st.xdims.append([xid])
            st.tdims.append([_Digit(int(n), xid)])
        return st

    def refine(self, dim: int, pos: int, major: int) -> None:
        """Split digit `pos` of T's dimension `dim` into (major, size // major);
        an X digit it carries is split the same way in X."""
        d = self.tdims[dim][pos]
        minor = d.size // major
        if d.x is None:
            self.tdims[dim][pos:pos + 1] = [_Digit(major), _Digit(minor)]
            return
        a, b = self.next_id, self.next_id + 1
        self.next_id += 2
        self.xsize[a], self.xsize[b] = major, minor
        for xd in self.xdims:
            if d.x in xd:
                k = xd.index(d.x)
                xd[k:k + 1] = [a, b]
        del self.xsize[d.x]
        self.tdims[dim][pos:pos + 1] = [_Digit(major, a), _Digit(minor, b)]


def _apply(st: _State, op: Op, pos: int, g: Graph) -> None:
    """T := op's output, where T is operand `pos` of op."""
    if op.kind == "elementwise":
        return
    if op.kind == "split":
        k, (a, _) = op.axis, op.sizes
        digits = st.tdims[k]
        prod, cut = 1, None
        for j, d in enumerate(digits):
            if prod == a:
                cut = j
                break
            if a % prod == 0 and d.size % (a // prod) == 0 and a // prod < d.size:
                st.refine(k, j, a // prod)
                cut = j + 1
                break
            prod *= d.size
        if cut is None and prod == a:
            cut = len(digits)
        if cut is None:  # not expressible on the digits: every X digit of the dimension becomes opaque
            for d in digits:
                if d.x is not None:
                    st.opaque.add(d.x)
            n = _prod(x.size for x in digits)
            st.tdims[k:k + 1] = [[_Digit(a)], [_Digit(n // a)]]
            return
        digits = st.tdims[k]
        st.tdims[k:k + 1] = [digits[:cut], digits[cut:]]
        return
    if op.kind == "merge":
        k = op.axis
        st.tdims[k:k + 2] = [st.tdims[k] + st.tdims[k + 1]]
        return
    if op.kind == "transpose":
        out: List[List[_Digit]] = [[] for _ in st.tdims]
        for i, j in enumerate(op.perm):
            out[j] = st.tdims[i]
        st.tdims = out
        return
    if op.kind == "broadcast":
        st.tdims.insert(op.axis, [_Digit(op.size)])
        return
    # contraction: T is operand `pos`
    ins, out = _parse_spec(op.spec)
    mine = ins[pos]
    of = {c: st.tdims[i] for i, c in enumerate(mine)}
    for c, digits in of.items():
        if c not in out:
            for d in digits:
                if d.x is not None:
                    st.reduced.add(d.x)
    shape = op.shape
    st.tdims = [of[c] if c in of else [_Digit(shape[i])] for i, c in enumerate(out)]


def _prod(xs) -> int:
    n = 1
    for x in xs:
        n *= x
    return n


def _preserving(st: _State, P: int) -> bool:
    """The check of Eq. 1 (see the module docstring)."""
    # where every X digit sits in T: (dimension, position)
    where: Dict[int, Tuple[int, int]] = {}
    for j, digits in enumerate(st.tdims):
        for p, d in enumerate(digits):
            if d.x is not None and d.x not in st.reduced and d.x not in st.opaque:
                where[d.x] = (j, p)
    for xd in st.xdims:
        n = _prod(st.xsize[x] for x in xd)
        if n % P:
            continue  # not a candidate for a mesh axis of P devices
        ok = False
        blocks = 1
        for p, x in enumerate(xd):
            loc = where.get(x)
            if loc is None or loc[1] != p or (p > 0 and loc[0] != where[xd[0]][0]):
                break
            blocks *= st.xsize[x]
            if blocks % P == 0:
                ok = True
                break
        if not ok:
            return False
    return True


# ------------------------------------------------------------ Algorithm 1 --

def build_parallel_blocks(g: Graph, P: int) -> List[List[str]]:
    """Phase 1 of ParallelBlock construction (Algorithm 1): the contractions in
    order of depth (then graph order); each one not yet grouped starts a block
    and grows it depth first through its users, taking the first user not yet
    grouped that keeps the block parallelism-preserving and continuing from it
    (the search returns after that user, as the algorithm states).  Operators
    left out of every block are not listed."""
    if P < 1:
        raise ValueError("P is a positive device count")
    depth = g.depth()
    order = {name: i for i, name in enumerate(g.ops)}
    contractions = sorted((o.name for o in g.ops.values() if o.kind == "contraction"),
                          key=lambda n: (depth[n], order[n]))
    grouped: set = set()
    blocks: List[List[str]] = []
    for s in contractions:
        if s in grouped:
            continue
        pb = [s]
        st = _State.start(g.ops[s].shape)
        cur = s
        while True:
            nxt = None
            for u in g.users(cur):
                if u in grouped or u in pb:
                    continue
                trial = _copy(st)
                _apply(trial, g.ops[u], g.ops[u].operands.index(cur), g)
                if _preserving(trial, P):
                    nxt, st = u, trial
                    break
            if nxt is None:
                break
            pb.append(nxt)
            cur = nxt
        grouped.update(pb)
        blocks.append(pb)
    return blocks


def _copy(st: _State) -> _State:
    return _State([list(x) for x in st.xdims], dict(st.xsize), [[_Digit(d.size, d.x) for d in ds] for ds in st.tdims],
                  set(st.reduced), set(st.opaque), st.next_id)


def is_parallelism_preserving(g: Graph, path: Sequence[str], P: int) -> bool:
    """The check of Eq. 1 for the chain `path`: the output of path[0] is X, each
    later operator reads the one before it, and the last one's output is
    compared with X."""
    st = _State.start(g.ops[path[0]].shape)
    for prev, u in zip(path, path[1:]):
        _apply(st, g.ops[u], g.ops[u].operands.index(prev), g)
    return _preserving(st, P)
