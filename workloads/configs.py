"""The five synthetic search workloads, named by shape.

Each stands in for the profiled tables of a transformer-like chain of
ParallelBlocks (12 blocks per layer, Sec. 4.1; tables reused across matched
layers, Sec. 2 overview step 4).  The paper's own profiles are not available,
so every table is drawn from `workloads.gen` with a fixed seed.

    chain_gpt_n24_k16      N=24   K=16  B=1    c,R ~ U[1e4,1e6)
    chain_gpt_n1152_k64    N=1152 K=64  B=256  c,R ~ U[1e4,1e7)
    mem_llama_n288_k32     N=288  K=32  B=16   c,R ~ U[1e4,1e6), mem ~ U{0..8},
                                               M=1024 buckets, budget_b = 1023-32b
    chain_wide_n512_k256   N=512  K=256 B=64   c,R ~ U[1e4,1e7), 25% of the
                                               off-diagonal R entries are 0
    scan_n4096_k512        N=4096 K=512 B=4    c,R ~ U[1e4,1e6)
    seg_gpt_n96_k81        N=96 segments, K=81 plans (4 blocks x 3 strategies),
                           B=256, c ~ U[4e4,4e7), boundary tables 2 x 3 x 3
                           ~ U[1e4,1e7) with a zero diagonal

All share 12 resharding tables with edge (i-1 -> i) using table i mod 12, and
R has a zero diagonal.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import gen

SEED_BASE = 2504005980
N_TABLES = 12


@dataclass(frozen=True)
class Config:
    idx: int
    name: str
    form: str          # "chain" | "mem" | "scan"
    N: int
    K: int
    B: int
    c_range: tuple
    r_range: tuple
    zero_frac_offdiag: float = 0.0
    M: int = 0
    mem_range: tuple = (0, 9)
    extra: dict = field(default_factory=dict)

    @property
    def seed(self) -> int:
        return SEED_BASE + self.idx

    @property
    def zeros(self) -> int:
        z = self.zero_frac_offdiag * self.K * (self.K - 1)
        if z != int(z):
            raise ValueError("zero fraction must give a whole count")
        return int(z)


CONFIGS = [
    Config(1, "chain_gpt_n24_k16", "chain", 24, 16, 1, (10_000, 1_000_000), (10_000, 1_000_000)),
    Config(2, "chain_gpt_n1152_k64", "chain", 1152, 64, 256, (10_000, 10_000_000), (10_000, 10_000_000)),
    Config(3, "mem_llama_n288_k32", "mem", 288, 32, 16, (10_000, 1_000_000), (10_000, 1_000_000), M=1024),
    Config(4, "chain_wide_n512_k256", "chain", 512, 256, 64, (10_000, 10_000_000), (10_000, 10_000_000),
           zero_frac_offdiag=0.25),
    Config(5, "scan_n4096_k512", "scan", 4096, 512, 4, (10_000, 1_000_000), (10_000, 1_000_000)),
    # segment-level search: 96 GPT-like layers as segments of 4 blocks x 3
    # strategies (81 plans), boundary resharding between the last and first
    # blocks (3 x 3), one table for the boundary after the first layer's
    # segment and one for the boundaries between repeated layers
    Config(6, "seg_gpt_n96_k81", "seg", 96, 81, 256, (40_000, 40_000_000), (10_000, 10_000_000),
           extra={"blocks": 4, "strategies": 3, "tables": 2}),
]

BY_NAME = {c.name: c for c in CONFIGS}
BY_IDX = {c.idx: c for c in CONFIGS}


def budgets(B: int) -> np.ndarray:
    """Budget (in memory buckets, inclusive) of search b: 1023 - 32 b."""
    return (1023 - 32 * np.arange(B)).astype(np.int32)


def make(cfg: Config | str | int, batch: int | None = None) -> dict:
    """Generate the arrays of a configuration.  `batch` < B keeps only the
    first searches (the per-search streams do not depend on B, so search b of
    a reduced batch equals search b of the full one)."""
    if isinstance(cfg, str):
        cfg = BY_NAME[cfg]
    elif isinstance(cfg, int):
        cfg = BY_IDX[cfg]
    B = cfg.B if batch is None else batch
    if cfg.form == "seg":
        P, S, E = cfg.extra["blocks"], cfg.extra["strategies"], cfg.extra["tables"]
        last, first = gen.digit_maps(P, S)
        redge = np.ones(cfg.N, np.int32)
        redge[:2] = 0
        return {
            "cost": gen.make_cost(cfg.seed, B, cfg.N, cfg.K, *cfg.c_range),
            "rbound": gen.make_rbound(cfg.seed, E, S, *cfg.r_range),
            "last": last,
            "first": first,
            "redge": redge,
        }
    out = {
        "cost": gen.make_cost(cfg.seed, B, cfg.N, cfg.K, *cfg.c_range),
        "rtab": gen.make_rtab(cfg.seed, N_TABLES, cfg.K, *cfg.r_range, zeros=cfg.zeros),
        "redge": gen.periodic_redge(cfg.N, N_TABLES),
    }
    if cfg.form == "mem":
        out["mem"] = gen.make_mem(cfg.seed, B, cfg.N, cfg.K, *cfg.mem_range)
        out["budget"] = budgets(B)
        out["M"] = cfg.M
    return out
