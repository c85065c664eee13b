"""ParallelBlock grouping (Sec. 3.2, Algorithm 1) with the parallelism-
preserving check of Eq. 1 over the element-level dependencies of Table 1.

The oracle evaluates Eq. 1 as its definition on dependency sets computed by
brute force from the operators' semantics; the product tracks the affine maps
symbolically.  Pins: hand cases whose answer follows from Sec. 3.1 directly
(element-wise chains, transposes, a reduced dimension, the self-attention
example of Sec. 3.1 with B and H divisible by the device count, the
reshape-BMM chain of Sec. 3.1 read with Table 1's row-major split), and
random graphs on which the two must agree block for block."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import frontend as OF
from paper_2504_00598_amd.parallel_blocks import Graph, build_parallel_blocks, is_parallelism_preserving


def both(g, P):
    got, want = build_parallel_blocks(g, P), OF.build_parallel_blocks(g, P)
    assert got == want
    return got


def check_path(g, path, P, expect):
    assert OF.path_preserving(g, path, P) == expect
    assert is_parallelism_preserving(g, path, P) == expect


def test_elementwise_chain_is_one_block():
    g = Graph()
    g.input("x", (4, 8)); g.input("w", (8, 8))
    g.contraction("mm", "ab,bc->ac", "x", "w")
    g.elementwise("gelu", "mm"); g.elementwise("drop", "gelu")
    g.input("res", (4, 8)); g.elementwise("add", "drop", "res")
    assert both(g, 2) == [["mm", "gelu", "drop", "add"]]
    check_path(g, ["mm", "gelu", "drop", "add"], 2, True)


def test_transpose_moves_dimensions_and_stays_preserving():
    g = Graph()
    g.input("x", (4, 8)); g.input("w", (8, 2))
    g.contraction("mm", "ab,bc->ac", "x", "w")
    g.transpose("t", "mm", (1, 0))
    check_path(g, ["mm", "t"], 2, True)
    assert both(g, 2) == [["mm", "t"]]


def test_reducing_a_partitioned_dimension_stops_the_block():
    """A contraction over dimension 1 of X: every output element depends on
    every index of that dimension, so no partition of it survives."""
    g = Graph()
    g.input("x", (4, 8)); g.input("w", (8, 8)); g.input("v", (8, 4))
    g.contraction("mm", "ab,bc->ac", "x", "w")
    g.contraction("mm2", "ab,bc->ac", "mm", "v")
    check_path(g, ["mm", "mm2"], 2, False)
    assert both(g, 2) == [["mm"], ["mm2"]]
    # with P = 4 only dimension 0 (4) and 1 (8) are candidates as well; with P = 3 none is
    check_path(g, ["mm", "mm2"], 3, True)


def test_self_attention_with_batch_and_heads_divisible():
    """Sec. 3.1: the attention block stays parallelism-preserving along the
    batch and head dimensions when both are divisible by the device count."""
    B, H, S, D = 2, 4, 3, 2
    g = Graph()
    g.input("q", (B, S, H, D)); g.input("k", (B, S, H, D)); g.input("v", (B, S, H, D))
    g.contraction("scores", "bshd,bthd->bhst", "q", "k")
    g.elementwise("softmax", "scores")
    g.contraction("ctx", "bhst,bthd->bshd", "softmax", "v")
    assert both(g, 2) == [["scores", "softmax", "ctx"]]
    # a sequence length divisible by P makes the reduced key dimension a candidate: the block stops
    g2 = Graph()
    g2.input("q", (B, 4, H, D)); g2.input("k", (B, 4, H, D)); g2.input("v", (B, 4, H, D))
    g2.contraction("scores", "bshd,bthd->bhst", "q", "k")
    g2.elementwise("softmax", "scores")
    g2.contraction("ctx", "bhst,bthd->bshd", "softmax", "v")
    assert both(g2, 2) == [["scores", "softmax"], ["ctx"]]


def test_reshape_bmm_chain_of_section_3_1():
    """The reshape, BMM, BMM, reshape chain of Sec. 3.1 ([A, B] -> [A, B1, B2]
    -> BMM contracting B1 -> BMM contracting C -> [A, B]).  With Table 1's
    row-major split, B1 is the leading factor of B, so a partition of B does
    not survive the first BMM; a partition of A survives the whole chain."""
    A, B1, B2, C = 6, 4, 4, 2

    def chain():
        g = Graph()
        g.input("x", (A, 8)); g.input("w", (8, B1 * B2))
        g.contraction("mm", "ab,bc->ac", "x", "w")
        g.split("r1", "mm", 1, (B1, B2))
        g.input("p1", (B2, C, B1)); g.contraction("bmm1", "abc,cdb->cad", "r1", "p1")
        g.input("p2", (B2, B1, C)); g.contraction("bmm2", "cad,cbd->abc", "bmm1", "p2")
        g.merge("r2", "bmm2", 1)
        return g

    g = chain()
    path = ["mm", "r1", "bmm1", "bmm2", "r2"]
    check_path(g, path, 3, True)            # only A (6) is a candidate for 3 devices
    assert both(g, 3) == [path]
    check_path(g, path, 2, False)           # B (16) is a candidate for 2 devices
    # with 2 devices every dimension is a candidate: the first BMM reduces B1 (the
    # leading factor of B), the second reduces C, and the final merge leaves B2 as
    # the trailing factor of a merged dimension, which contiguous blocks split
    assert both(g, 2) == [["mm", "r1"], ["bmm1"], ["bmm2"]]


def test_first_qualifying_user_only():
    """The search continues from the first user that keeps the block
    preserving; later users of the same operator start no branch of it."""
    g = Graph()
    g.input("x", (4, 4)); g.input("w", (4, 4))
    g.contraction("mm", "ab,bc->ac", "x", "w")
    g.elementwise("a1", "mm"); g.elementwise("a2", "mm")
    assert both(g, 2) == [["mm", "a1"]]


def _random_graph(rs, n_ops):
    g = Graph()
    g.input("x0", (2, 4))
    g.input("w0", (4, 4))
    g.contraction("c0", "ab,bc->ac", "x0", "w0")
    names = ["c0"]
    letters = "abcdefgh"
    for n in range(n_ops):
        src = names[int(rs.integers(0, len(names)))] if rs.random() < 0.4 else names[-1]
        shp = g.ops[src].shape
        kind = rs.choice(["elementwise", "split", "merge", "transpose", "broadcast", "contraction", "contraction"])
        name = f"o{n}"
        numel = int(np.prod(shp))
        try:
            if kind == "elementwise":
                g.elementwise(name, src)
            elif kind == "split":
                k = int(rs.integers(0, len(shp)))
                if shp[k] < 4 or len(shp) >= 4:
                    continue
                a = 2 if rs.random() < 0.5 else shp[k] // 2
                g.split(name, src, k, (a, shp[k] // a))
            elif kind == "merge":
                if len(shp) < 2 or numel > 64:
                    continue
                g.merge(name, src, int(rs.integers(0, len(shp) - 1)))
            elif kind == "transpose":
                g.transpose(name, src, tuple(int(x) for x in rs.permutation(len(shp))))
            elif kind == "broadcast":
                if len(shp) >= 4 or numel > 32:
                    continue
                g.broadcast(name, src, int(rs.integers(0, len(shp) + 1)), 2)
            else:
                mine = letters[:len(shp)]
                keep = [c for c in mine if rs.random() < 0.7]
                new = [] if rs.random() < 0.5 or len(keep) >= 3 else ["z"]
                out = list(keep) + new
                rs.shuffle(out)
                pshape_letters = [c for c in mine if c not in keep or rs.random() < 0.3] + new
                if not pshape_letters:
                    pshape_letters = [mine[0]]
                psh = tuple(shp[mine.index(c)] if c in mine else 2 for c in pshape_letters)
                if not out or int(np.prod([shp[mine.index(c)] if c in mine else 2 for c in out])) > 128:
                    continue
                g.input(f"p{n}", psh)
                g.contraction(name, f"{mine},{''.join(pshape_letters)}->{''.join(out)}", src, f"p{n}")
        except ValueError:
            continue
        names.append(name)
    return g


@pytest.mark.parametrize("seed", range(100))
def test_random_graphs_agree_with_the_brute_force(seed):
    rs = np.random.default_rng([81, seed])
    g = _random_graph(rs, int(rs.integers(3, 9)))
    for P in (2, 4):
        both(g, P)
